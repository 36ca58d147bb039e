// Sparse attention over an index list (Eq. 3 of "LongCat Sparse Attention", arXiv 2608.01662)
// for gfx950: MLA absorbed mode (64 heads, latent rows of 576 = 512 + 64 bf16, V = first 512
// columns) and MQA-128 (16 heads, separate K and V of 128).
//
// Both kernels compute S^T = K Q^T (keys on the MFMA rows, heads on the columns) so that in the
// accumulator layout each lane holds several tokens of one head per block: the per-head softmax
// max and sum are in-lane reductions plus two lane exchanges, and the exponentiated scores are in
// the B-operand layout of the product O^T += V^T P^T (MQA: in registers; MLA: written head-major
// to LDS for the value waves). V^T reaches the A-operand layout through ds_read_b64_tr_b16 (a
// 16 x 4 transpose read on gfx950), so V is stored once, token-major, in the same LDS tile as K.
//
// Online softmax in base 2 with a lazily updated reference maximum: the accumulators are only
// rescaled when a head's running maximum grows by more than 2^8, which keeps every
// exponentiated score in (0, 256] and leaves the result exact up to rounding.
#include "device.hpp"
#include "launch.hpp"

namespace lsa {

constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kLazy = 8.0f;  // rescale when the max grows by more than this (log2 units)

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ u32x4 tr16_pair(const uint8_t* pa, const uint8_t* pb) {
  const s16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(pa));
  const s16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(pb));
  const u32x2 a2 = __builtin_bit_cast(u32x2, va), b2 = __builtin_bit_cast(u32x2, vb);
  return u32x4{a2.x, a2.y, b2.x, b2.y};
}

// ============================================================================ MLA 64 x 576 / 512
// One workgroup = 8 waves = one query row (or one split of its index list), two waves per SIMD.
// The waves split the work by role:
//   * scorer w (w < 4) computes S^T for tokens 16 (w & 1) .. + 15 of every tile and the 32 heads
//     32 (w >> 1) .. + 31 (two 16x16x32 head blocks sharing each K operand, so that every K byte
//     is read by two scorers per tile) over all 576 dims, does the online softmax of its token
//     half and leaves P (bf16, head-major) and the reference maximum it used in an LDS slot;
//   * value wave w + 4, one tile behind, accumulates O^T += V^T P^T for all 64 heads and value
//     columns 128 w .. + 127 on 32x32x16 products (dims on the rows, heads on the columns): each V
//     operand feeds two head blocks, and every V byte is read once per tile.
// The two token halves of a head keep their own reference maxima. A scorer adopts the other
// half's reference of the previous tile when that is larger, so the two differ only in the tile
// after one of them moved; the value wave then brings the lower half's P (rounded to bf16 a second
// time) and its accumulators to the larger one. No score is split across waves, so the only
// synchronisation is one barrier per tile: at barrier it, tile it has landed, the scorers have
// written P of tile it - 1 and the value waves are done with tile it - 2. Three tile buffers
// rotate (tile it scored, tile it - 1 in the value products, tile it + 1 loading); the value waves
// issue the loads and the P slots alternate by tile parity. A scorer holds 144 Q-operand
// registers, a value wave 128 accumulator registers; the two roles run separate loops with the
// same barrier sequence, so that their registers share the file.
//
// The row's index list is validated once into LDS (-1 for entries to skip). Tiles of 32 gathered
// latent rows are moved by direct global->LDS loads. Tile layout: 1 KB blocks of 8 tokens x 8
// chunks (chunk c = dims 8c..8c+7): token t = 8o + j, chunk c sits in block 9o + c / 8 at 16-byte
// slot 8j + ((c % 8) ^ mla_swz(o, j)), mla_swz(o, j) = 4 j1 + 2 j2 + (o & 1) with j1, j2 bits 1 and
// 2 of j. One direct load fills one block, eight consecutive lanes taking one whole 128-byte line
// of one row (8 rows per load), and the XOR keeps the K-operand reads (16 tokens, one chunk per
// 16 lanes) and the value waves' transposed V reads (per 32 lanes, 4 token rows x 64 bytes: rows
// 4r and 4r + 2, which share a half of the banks, land in opposite halves of the slots) free of
// LDS bank conflicts (checked on the host against 64 banks of 4 bytes, 32 lanes per cycle). The K reads still take the LDS's
// slower path (about 120 instead of 200 bytes per clock): a ds_read_b128 runs at full rate only
// when each 16-lane quarter reads one aligned 256-byte segment, which a token-major tile cannot
// offer for 16 tokens of one chunk; layouts that do (chunk-major) need loads that touch 16 or 32
// rows each, and those measured slower overall.
//
// Before the role split, wave (hq, kw) computed half of the dims of S for its 16 heads and the
// pair summed their partials through LDS behind a second barrier per tile (74 ms per layer at
// L = 128K against 62 ms for the split with 16-head value waves, same LDS bytes otherwise): the
// cost was the extra synchronisation of the eight waves, not the bytes exchanged. 32-head value
// waves then halved the transposed V reads (60 ms), scorers split by tokens instead of heads
// halved the K reads (56 ms), and 64-head value waves halved the V reads again (55 ms).
constexpr int kMlaT = 32;
constexpr int kMlaTile = 36 * 1024;  // 72 chunks x 32 tokens x 16 bytes
constexpr int kMlaBufs = 3;          // tile buffers: scored, in the value products, loading
constexpr int kMlaLoads = 9;         // direct loads per value wave per tile (36 x 1 KB)
constexpr int kMlaPHead = 80;        // bytes per head in a P slot: 32 bf16 tokens + 16 B of padding
constexpr int kMlaPSlot = 64 * kMlaPHead + 2 * 64 * 4;  // per tile parity: P of 64 heads + the reference maxima of both token halves
__device__ __forceinline__ int mla_swz(int o, int j) { return ((j & 2) << 1) | ((j & 4) >> 1) | (o & 1); }
constexpr int kMlaHalf = 18 * 1024;  // the second 16 tokens of a tile start 18 blocks later
constexpr int kMlaIdCap = 8192;      // index-list entries staged in LDS at a time
// Nine direct loads of one 1152-byte row piece per lane: load k reads the 16 bytes at src + 128 k
// and writes LDS bytes [lds + 1024 k + 16 lane, +16). The loads share one address and carry
// 128 k as their immediate offset, which these loads add to the LDS address as well, so M0 steps
// by 1024 - 128 per load. Written as one asm block so that the compiler does not see LDS being
// written by vector-memory loads: it would otherwise drain every such load in flight before any
// later LDS read it cannot prove disjoint; callers order the loads with explicit vmcnt waits and
// barriers. M0, which holds the LDS address of the loads, is saved and restored; the s_nop after
// each write of M0 is the wait state before a load may read it.
__device__ __forceinline__ void lds_dma_row9(const uint8_t* src, uint32_t lds) {
  uint32_t save;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_add_u32 m0, m0, 0x380\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off offset:128\n\t"
      "s_add_u32 m0, m0, 0x380\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off offset:256\n\t"
      "s_add_u32 m0, m0, 0x380\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off offset:384\n\t"
      "s_add_u32 m0, m0, 0x380\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off offset:512\n\t"
      "s_add_u32 m0, m0, 0x380\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off offset:640\n\t"
      "s_add_u32 m0, m0, 0x380\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off offset:768\n\t"
      "s_add_u32 m0, m0, 0x380\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off offset:896\n\t"
      "s_add_u32 m0, m0, 0x380\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off offset:1024\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(save)
      : "v"(src), "s"(lds)
      : "memory", "scc");
}

// The maxima of x and of y over the four 16-lane rows (lanes l, l ^ 16, l ^ 32, l ^ 48), sharing
// the lane swaps: the first swap leaves rows (x0, y0, x2, y2) and (x1, y1, x3, y3), the second
// (row halves) rows x, y, x, y of the full maxima, the last hands each lane both.
__device__ __forceinline__ void max4_xor16_32_pair(float& x, float& y) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(y), false, false);
  const float z = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(z), __float_as_uint(z), false, false);
  const float w = fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
  const auto c = __builtin_amdgcn_permlane16_swap(__float_as_uint(w), __float_as_uint(w), false, false);
  x = __uint_as_float(c[0]);
  y = __uint_as_float(c[1]);
}
constexpr float kNoRef = -3.40282347e38f;  // reference maximum before a head's first score (finite, so
                                           // exp2(s - m) needs no guard: masked scores are -inf)

// eight bf16 scaled by f (rounded to nearest even again)
__device__ __forceinline__ u32x4 scale_bf16x8(u32x4 v, float f) {
  u32x4 r;
#pragma unroll
  for (int k = 0; k < 4; ++k)
    r[k] = pack_bf16x2(__uint_as_float(v[k] << 16) * f, __uint_as_float(v[k] & 0xFFFF0000u) * f);
  return r;
}

// Run form of an index list: runs [start, start + len) of cache rows, in list order. Thread t of
// the 512 takes the contiguous block of runs [t U, t U + U), U = ceil(n_runs / 512).
struct RunBlock {
  const int32_t* base;  // this row's runs (int32 pairs)
  int b, e;             // this thread's runs
};
__device__ __forceinline__ RunBlock run_block(const AttnGeom& a, int64_t row) {
  int nr = a.run_count[row];
  nr = nr < 0 ? 0 : (nr > a.k_cap ? a.k_cap : nr);
  const int u = (nr + 511) / 512;
  const int b = (int)threadIdx.x * u;
  return RunBlock{a.runs + row * a.k_cap * 2, b < nr ? b : nr, b + u < nr ? b + u : nr};
}
// Length of a run, clamped to [0, cap]: a run longer than the list capacity ends the list anyway.
__device__ __forceinline__ int run_len(int l, int cap) { return l < 0 ? 0 : (l > cap ? cap : l); }
// Runs [r0, r0 + 4) of this thread's block, loaded together (zero-length past the block's end).
__device__ __forceinline__ void load_runs4(const RunBlock& rb, int r0, int2 (&x)[4]) {
#pragma unroll
  for (int k = 0; k < 4; ++k)
    x[k] = r0 + k < rb.e ? *reinterpret_cast<const int2*>(rb.base + 2 * (r0 + k)) : int2{0, 0};
}
constexpr int kRunShort = 4;   // runs longer than this are expanded by the whole block
constexpr int kRunQueue = 128; // long runs queued per staging pass (more are expanded by their owner)
// Exclusive prefix over the 512 threads of v (list entries before this thread's runs) and the total.
__device__ __forceinline__ int64_t block_prefix512(int64_t v, int64_t* wtot, int64_t& total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int64_t inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t t = __shfl_up(inc, o);
    if (lane >= o) inc += t;
  }
  if (lane == 63) wtot[wv] = inc;
  __syncthreads();
  int64_t base = 0;
  total = 0;
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    base += x < wv ? wtot[x] : 0;
    total += wtot[x];
  }
  __syncthreads();
  return base + inc - v;
}

// WIN: the window branch of the split attention as a query-tiled kernel (Sec. 4.1.1): a workgroup
// takes two consecutive query rows t0, t0 + 1 and heads 32 blockIdx.y .. + 31, and walks the
// contiguous cache rows of the union of their windows, [t0 - k_swa + 1, t0 + 1], once: every tile
// is loaded once into LDS for both rows. Scorer w4 works on row t0 + (w4 >> 1), heads
// 32 blockIdx.y .. + 31 and tokens 16 (w4 & 1) .. of every tile, value wave w4 + 4 on both rows,
// heads 32 blockIdx.y .. + 31 and value columns 128 w4 ..; each row masks the tokens outside its
// own window.
// Writes the fp32 partial of split a.part.
// (Two rows of 64 heads would hold 2 x (73.7 KB of Q operand + 131 KB of fp32 accumulators), 80%
// of a CU's 512 KB register file, before any operand; tiling 2 rows x 32 heads keeps the 64 query
// vectors per tile of the list kernel.)
template <bool SPLIT, bool WIN = false>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void mla_attn_kernel(AttnGeom a) {
  static_assert(!WIN || SPLIT, "the window kernel writes partials");
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kMlaBufs * kMlaTile + 2 * kMlaPSlot];
  __shared__ int32_t ids[WIN ? 1 : kMlaIdCap];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int i16 = lane & 15, g = lane >> 4;
  const int w4 = wv & 3;  // scorer / value-wave pair
  const bool scorer = wv < 4;
  // WIN: item = row pair, pair w4 on row 2 item + (w4 >> 1); the second row of a pair past n_rows
  // (odd count) computes nothing it writes
  const int64_t item = xcd_band(blockIdx.x, WIN ? (a.n_rows + 1) / 2 : a.n_rows);
  const int64_t wrow = WIN ? 2 * item + (w4 >> 1) : item;
  const bool row_ok = wrow < a.n_rows;
  const int64_t row = row_ok ? wrow : a.n_rows - 1;
  const int split = SPLIT ? (a.part >= 0 ? a.part : (int)blockIdx.y) : 0;
  __shared__ int64_t rtot[8];
  __shared__ int32_t roff[512];   // run form: list position of each thread's first run (clamped)
  __shared__ int4 rq[kRunQueue];  // run form: (start, offset into the run, ids slot, entries)
  __shared__ int rq_n;
  int cnt;
  if (WIN) {
    cnt = 0;  // (unused: the window is generated)
  } else if (a.runs) {  // the list length is the sum of the run lengths (at most k_cap entries are used)
    const RunBlock rb = run_block(a, row);
    int64_t mine = 0;
    for (int r0 = rb.b; r0 < rb.e; r0 += 4) {
      int2 x[4];
      load_runs4(rb, r0, x);
#pragma unroll
      for (int k = 0; k < 4; ++k) mine += run_len(x[k].y, a.k_cap);
    }
    int64_t total;
    const int64_t off = block_prefix512(mine, rtot, total);
    roff[threadIdx.x] = (int)(off < 0x7fffffff ? off : 0x7fffffff);  // read back by this thread only
    cnt = (int)(total > a.k_cap ? a.k_cap : total);
  } else {
    cnt = a.count[row];
    cnt = cnt < 0 ? 0 : (cnt > a.k_cap ? a.k_cap : cnt);
  }
  int s0 = SPLIT && a.part < 0 ? split * a.split_len : 0;
  int s1 = SPLIT && a.part < 0 ? (cnt < s0 + a.split_len ? cnt : s0 + a.split_len) : cnt;
  int64_t win0 = -1;  // first cache row of the window part (contiguous rows, no list)
  // WIN: this wave's row window [w_lo, w_hi] (empty for a skipped row) and the pair's union
  int64_t w_lo = 0, w_hi = -1, u_last = -1;
  if (WIN) {
    const int64_t t0 = a.q_pos0 + 2 * item;
    const int64_t t1 = a.q_pos0 + (2 * item + 1 < a.n_rows ? 2 * item + 1 : 2 * item);
    const int64_t t = a.q_pos0 + row;
    int c = a.count[row];
    if (row_ok && c > 0) {  // an empty list (a skipped row) has no window either
      w_hi = t;
      w_lo = t - a.k_swa + 1 > 0 ? t - a.k_swa + 1 : 0;
    }
    win0 = t0 - a.k_swa + 1 > 0 ? t0 - a.k_swa + 1 : 0;
    u_last = t1 < a.n_kv_rows - 1 ? t1 : a.n_kv_rows - 1;
    s0 = 0;
    s1 = (int)(t1 - win0 + 1);
  } else if (a.part >= 0) {
    const int64_t t = a.q_pos0 + row;
    const int nwin = (int)(a.k_swa < t + 1 ? a.k_swa : t + 1);
    if (a.part == 0) {
      s1 = cnt - nwin > 0 ? cnt - nwin : 0;
    } else {
      s1 = cnt > 0 ? nwin : 0;  // an empty list (a skipped row) has no window either
      win0 = t - nwin + 1;
    }
  }
  const int n = s1 > s0 ? s1 - s0 : 0;
  const int32_t* slots = a.rows ? a.rows + row * a.k_cap + s0 : nullptr;  // list form (unused with runs)
  const uint8_t* kvb = reinterpret_cast<const uint8_t*>(a.kv);
  uint8_t* const pslots = lds + kMlaBufs * kMlaTile;
  // P slots: head-major [2 scorer pairs][32 heads][32 tokens] bf16, then the reference maxima
  // [2 token halves][64 (pair, local head)]; scorer w4 writes tokens 16 (w4 & 1) .. of the 32
  // heads of pair w4 >> 1, every value wave reads all 64
  const int pair = w4 >> 1;
  __shared__ float fin[2 * 2 * 64];           // per (token half, pair, local head): reference max and sum

  constexpr int kPass = WIN ? (1 << 30) : kMlaIdCap;  // the window needs no staged list
  // list entries [c0, c0 + nc) -> LDS, validated (-1 = skip; the last tile is padded with -1)
  auto stage = [&](int c0, int nc, int ntiles) {
    if (a.runs && threadIdx.x == 0) rq_n = 0;  // the previous pass's readers passed a barrier since
    __syncthreads();  // the previous chunk's readers of `ids` are done
    if (a.runs) {
      // list entries [s0 + c0, s0 + c0 + nc) from the runs (runs partition the list, so every entry
      // is written once): each thread writes the entries of its own short runs that fall in this
      // chunk and queues the longer ones, which the whole block then writes, 512 entries at a time
      const RunBlock rb = run_block(a, row);
      const int64_t lo = (int64_t)s0 + c0, hi = lo + nc;
      int64_t off = roff[threadIdx.x];
      for (int r0 = rb.b; r0 < rb.e && off < hi; r0 += 4) {
        int2 x[4];
        load_runs4(rb, r0, x);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const int64_t len = run_len(x[k].y, a.k_cap);
          const int64_t p0 = off > lo ? off : lo, p1 = off + len < hi ? off + len : hi;
          if (p1 > p0) {
            int q = kRunQueue;
            if (p1 - p0 > kRunShort) q = atomicAdd(&rq_n, 1);
            if (q < kRunQueue) {
              rq[q] = int4{x[k].x, (int)(p0 - off), (int)(p0 - lo), (int)(p1 - p0)};
            } else {
              for (int64_t pp = p0; pp < p1; ++pp) {
                const int64_t v = (int64_t)x[k].x + (pp - off);
                ids[pp - lo] = (v >= 0 && v < a.n_kv_rows) ? (int)v : -1;
              }
            }
          }
          off += len;
        }
      }
      for (int i = nc + (int)threadIdx.x; i < ntiles * kMlaT; i += 512) ids[i] = -1;  // pad the last tile
      __syncthreads();
      const int nq = rq_n < kRunQueue ? rq_n : kRunQueue;
      for (int qi = 0; qi < nq; ++qi) {
        const int4 e = rq[qi];
        for (int i = (int)threadIdx.x; i < e.w; i += 512) {
          const int64_t v = (int64_t)e.x + e.y + i;
          ids[e.z + i] = (v >= 0 && v < a.n_kv_rows) ? (int)v : -1;
        }
      }
    } else {
      constexpr int U = kMlaIdCap / 512;
      int v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = (int)threadIdx.x + 512 * u;
        v[u] = i < nc ? (win0 >= 0 ? (int)(win0 + c0 + i) : slots[c0 + i]) : -1;
      }
      if (a.page_table) {  // paged cache: position -> cache row through the sequence's page table
        const int32_t* tab = a.page_table + (row / a.rows_per_seq) * a.max_pages;
        const int kvp = a.kv_page;
        const bool p2 = (kvp & (kvp - 1)) == 0;
        const int lg = __ffs(kvp) - 1;
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int pos = v[u];
          if (pos >= 0) {
            const int pg = p2 ? pos >> lg : pos / kvp;
            const int64_t ph = pg < a.max_pages ? tab[pg] : -1;
            const int64_t cr = ph * kvp + (pos - pg * kvp);
            v[u] = (ph >= 0 && cr < a.n_kv_rows) ? (int)cr : -1;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = (int)threadIdx.x + 512 * u;
        if (i < ntiles * kMlaT) ids[i] = (v[u] >= 0 && (int64_t)v[u] < a.n_kv_rows) ? v[u] : -1;
      }
    }
    __syncthreads();
  };
  // cache row of token `tok` of tile `tile` (WIN: contiguous rows; positions past the union re-read
  // its last row, masked), -1 for a skipped entry
  auto tile_row = [&](int tile, int tok) -> int {
    if constexpr (WIN) {
      const int64_t p = win0 + (int64_t)tile * kMlaT + tok;
      return (int)(p < u_last ? p : u_last);
    } else {
      return ids[tile * kMlaT + tok];
    }
  };

  if (scorer) {
    // scorer w4 takes tokens 16 th .. + 15 of every tile for the 32 heads of its pair
    const int th = w4 & 1;
    const int hbase = WIN ? 32 * (int)blockIdx.y : 32 * pair;
    // Q^T as the B operand of S^T = K Q^T: column = head 16 nb + i16, k-step s covers dims 32s + 8g .. +7
    u32x4 qb[2][18];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const u32x4* qp = reinterpret_cast<const u32x4*>(a.q + (row * 64 + hbase + 16 * nb + i16) * 576 + 8 * g);
#pragma unroll
      for (int s = 0; s < 18; ++s) qb[nb][s] = qp[4 * s];
    }
    // K operand of k-step s: token 16 th + i16 = 8(2th + i16/8) + (i16 % 8), chunk
    // 4s + g = 8 (s/2) + 4 (s % 2) + g: one base offset for even and one for odd s, the rest an
    // immediate (s/2 blocks)
    const int ksw = mla_swz(i16 >> 3, i16 & 7);
    const int k_row = th * kMlaHalf + 9 * (i16 >> 3) * 1024 + 8 * (i16 & 7) * 16;
    const int k_even = k_row + ((0 + g) ^ ksw) * 16, k_odd = k_row + ((4 + g) ^ ksw) * 16;
    const int lj = lane & 31;  // token of this lane's validity bit in the softmax mask
    float m[2] = {kNoRef, kNoRef}, l[2] = {0.f, 0.f};
    for (int c0 = 0; c0 < n; c0 += kPass) {
      const int nc = n - c0 < kPass ? n - c0 : kPass;
      const int ntiles = (nc + kMlaT - 1) / kMlaT;
      if constexpr (!WIN) stage(c0, nc, ntiles);
      __syncthreads();
      uint32_t cur_off = 0;
      for (int it = 0; it <= ntiles; ++it) {
        // tile it has landed; this scorer's P writes of tile it - 1 are complete
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        const uint8_t* tb = lds + __builtin_amdgcn_readfirstlane(cur_off);
        cur_off = cur_off + kMlaTile == kMlaBufs * kMlaTile ? 0 : cur_off + kMlaTile;
        if (it == ntiles) continue;  // (the value waves' last tile)
        // issued first, so that their LDS round trips overlap the products: this lane's list entry
        // of the tile (softmax mask) and the other token half's reference maxima of tile it - 1
        // (adopted when larger)
        int idv = 0;
        if constexpr (!WIN) idv = ids[it * kMlaT + lj];
        float mp[2] = {-INFINITY, -INFINITY};
        if (it > 0) {
          const uint8_t* pr = pslots + ((it - 1) & 1) * kMlaPSlot + 64 * kMlaPHead + (1 - th) * 256;
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) mp[nb] = *reinterpret_cast<const float*>(pr + 4 * (32 * pair + 16 * nb + i16));
        }
        // S^T over all 576 dims: K operands in batches of KB, the next batch requested before the
        // products of the current one; every K operand feeds both head blocks
        constexpr int KB = 3;
        f32x4 sacc[2] = {f32x4{}, f32x4{}};
        u32x4 ka[2][KB];
#pragma unroll
        for (int s6 = 0; s6 < KB; ++s6)
          ka[0][s6] = *reinterpret_cast<const u32x4*>(tb + ((s6 & 1) ? k_odd : k_even) + (s6 >> 1) * 1024);
#pragma unroll
        for (int bt = 0; bt < 18 / KB; ++bt) {
          if (bt + 1 < 18 / KB) {
#pragma unroll
            for (int s6 = 0; s6 < KB; ++s6) {
              const int s = KB * (bt + 1) + s6;
              ka[(bt + 1) & 1][s6] = *reinterpret_cast<const u32x4*>(tb + ((s & 1) ? k_odd : k_even) + (s >> 1) * 1024);
            }
          }
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int s6 = 0; s6 < KB; ++s6)
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) sacc[nb] = mfma16(ka[bt & 1][s6], qb[nb][KB * bt + s6], sacc[nb]);
          __builtin_amdgcn_sched_barrier(0);
        }
        // online softmax (base 2); lane holds tokens 16 th + 4g + r of heads 16 nb + i16
        uint32_t vmask;
        if constexpr (WIN) {
          const int64_t p = win0 + (int64_t)it * kMlaT + lj;
          vmask = (uint32_t)__ballot(p >= w_lo && p <= w_hi);
        } else {
          vmask = (uint32_t)__ballot(idv >= 0);
        }
        const uint32_t hmask = (vmask >> (16 * th)) & 0xFFFFu;
        if (hmask != 0xFFFFu) {  // partial or skipped tokens: mask them
#pragma unroll
          for (int nb = 0; nb < 2; ++nb)
#pragma unroll
            for (int r = 0; r < 4; ++r) sacc[nb][r] = ((hmask >> (4 * g + r)) & 1u) ? sacc[nb][r] : -INFINITY;
        }
        uint8_t* slot = pslots + (it & 1) * kMlaPSlot;
        float smx[2];
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) smx[nb] = fmaxf(fmaxf(sacc[nb][0], sacc[nb][1]), fmaxf(sacc[nb][2], sacc[nb][3]));
        max4_xor16_32_pair(smx[0], smx[1]);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          const float mx = smx[nb] * a.scale_log2;  // scale > 0: max commutes with scaling
          // the reference maximum moves when a head's maximum grows by more than 2^8, or to the
          // other half's reference when that is larger; the value wave reconciles the two halves
          float tgt = mx > m[nb] + kLazy ? mx : m[nb];
          tgt = fmaxf(tgt, mp[nb]);
          const bool up = tgt > m[nb];
          if (__ballot(up)) {  // rare once a row's scores have settled
            l[nb] = up ? l[nb] * fast_exp2(m[nb] - tgt) : l[nb];
            m[nb] = up ? tgt : m[nb];
          }
          float p[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            p[r] = fast_exp2(fmaf(sacc[nb][r], a.scale_log2, -m[nb]));  // -inf -> 0
            l[nb] += p[r];
          }
          // P of tokens 16 th + 4g .. + 3, bf16, into the head's row of the slot
          const int lh = 32 * pair + 16 * nb + i16;  // (pair, local head)
          *reinterpret_cast<u32x2*>(slot + lh * kMlaPHead + 32 * th + 8 * g) = u32x2{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3])};
          if (g == 0) *reinterpret_cast<float*>(slot + 64 * kMlaPHead + th * 256 + 4 * lh) = m[nb];
        }
      }
    }
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const float lt = sum4_xor16_32(l[nb]);
      if (g == 0) {
        const int lh = 32 * pair + 16 * nb + i16;
        fin[2 * (64 * th + lh)] = m[nb];
        fin[2 * (64 * th + lh) + 1] = lt;
      }
    }
    __syncthreads();
    return;
  }

  // ---- value wave w4: O^T += V^T P^T for all 64 (pair, local head) columns and value columns
  // 128 w4 .. + 127, one tile behind the scorers, on 32x32x16 products (dims on the rows, heads on
  // the columns, 16 tokens per k-step): every V operand feeds both head blocks, and every V byte is
  // read by one value wave per tile. A operand of value block c (dims 128 w4 + 32 c ..), k-step ks:
  // lane l holds dim l % 32, tokens 16 ks + 8 (l / 32) + 0..7, from two transposed reads; in
  // 16-lane group G = l / 16, source lane s of read r supplies token 16 ks + 8 (G / 2) + 4 r + s / 4,
  // dims 128 w4 + 32 c + 16 (G % 2) + 4 (s % 4) .. + 3: chunk 16 w4 + 4 c + 2 (G % 2) + (s % 4) / 2,
  // i.e. block 9 (2 ks + G / 2) + 2 w4 + c / 2, chunk 4 (c % 2) + 2 (G % 2) + (s % 4) / 2 of it. The
  // swizzle depends on the token row and o % 2 only, so there is one base offset per (r, c % 2) and
  // the rest is an immediate (ks * 18 KB, (c / 2) KB).
  const int G = lane >> 4, sl = lane & 15;
  int v_off[2][2];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int par = 0; par < 2; ++par) {
      const int tk = 8 * (G >> 1) + 4 * r + (sl >> 2), o = tk >> 3, j = tk & 7;
      const int ch = 4 * par + 2 * (G & 1) + ((sl >> 1) & 1);  // chunk within the block 9 o + 2 w4 + c / 2
      v_off[r][par] = (9 * o + 2 * w4) * 1024 + (8 * j + (ch ^ mla_swz(o, j))) * 16 + (sl & 1) * 8;
    }
  const int oj = lane & 31;  // local head of this lane's accumulator column in each head block
  f32x16 o[8];               // block 4 hb + c: heads 32 hb .., dims 128 w4 + 32 c ..
#pragma unroll
  for (int c = 0; c < 8; ++c) o[c] = f32x16{};
  float m_o[2] = {-INFINITY, -INFINITY};  // reference maxima of the accumulators
  // Direct load k of value wave w4 fills block 9 w4 + k (tokens 8 w4.., chunks 8k..): lane 8j + u
  // takes token 8 w4 + j, chunk 8k + (u ^ mla_swz(w4, j)), 16 bytes of one 128-byte line per lane.
  const int dj = lane >> 3;
  const int dma_tok = 8 * w4 + dj;
  const int64_t dma_col = ((lane & 7) ^ mla_swz(w4, dj)) * 16;
  auto issue = [&](int r, uint32_t buf_off) {
    lds_dma_row9(kvb + (int64_t)(r > 0 ? r : 0) * 1152 + dma_col, lds_addr(lds + buf_off + w4 * (kMlaLoads * 1024)));
  };
  for (int c0 = 0; c0 < n; c0 += kPass) {
    const int nc = n - c0 < kPass ? n - c0 : kPass;
    const int ntiles = (nc + kMlaT - 1) / kMlaT;
    if constexpr (!WIN) stage(c0, nc, ntiles);
    __syncthreads();
    if (ntiles > 0) issue(tile_row(0, dma_tok), 0);
    int nrow = ntiles > 1 ? tile_row(1, dma_tok) : -1;  // row of this lane's next load, read a tile ahead
    // buffer byte offsets rotated as wave-uniform scalars: tile it - 1 (read now), it, it + 1
    uint32_t prev_off = 2 * kMlaTile, cur_off = 0, next_off = kMlaTile;
    u32x4 va[4][2];  // V operands of tile it - 1, read in the previous iteration
    for (int it = 0; it <= ntiles; ++it) {
      // tile it has landed; the scorers' P of tile it - 1 is in its slot; tile it - 2 is free
      asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
      if (it + 1 < ntiles) issue(nrow, next_off);
      if (it + 2 < ntiles) nrow = tile_row(it + 2, dma_tok);
      const uint32_t t0 = prev_off;
      prev_off = cur_off;
      cur_off = next_off;
      next_off = t0;
      // V operands of tile it (landed), for the products of the next iteration: four value
      // blocks, both k-steps
      auto read_v = [&]() {
        const uint8_t* tp = lds + __builtin_amdgcn_readfirstlane(prev_off);
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            const uint8_t* b0 = tp + v_off[0][c & 1] + ks * kMlaHalf + (c >> 1) * 1024;
            const uint8_t* b1 = tp + v_off[1][c & 1] + ks * kMlaHalf + (c >> 1) * 1024;
            va[c][ks] = tr16_pair(b0, b1);
          }
      };
      if (it == 0) {  // (nothing scored yet)
        read_v();
        continue;
      }
      const uint8_t* slot = pslots + ((it - 1) & 1) * kMlaPSlot;
      // the tile's LDS reads first (reference maxima, P; V was read a tile ahead), then the checks
      float mA[2], mB[2];
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        mA[hb] = *reinterpret_cast<const float*>(slot + 64 * kMlaPHead + 4 * (32 * hb + oj));
        mB[hb] = *reinterpret_cast<const float*>(slot + 64 * kMlaPHead + 256 + 4 * (32 * hb + oj));
      }
      // B operand P^T of head block hb, k-step ks: head 32 hb + oj, tokens 16 ks + 8 (l / 32) .. + 7
      u32x4 pb[2][2];
#pragma unroll
      for (int hb = 0; hb < 2; ++hb)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
          pb[hb][ks] = *reinterpret_cast<const u32x4*>(slot + (32 * hb + oj) * kMlaPHead + 32 * ks + 16 * (lane >> 5));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        const float mn = fmaxf(mA[hb], mB[hb]);  // >= m_o: the references never decrease
        if (__ballot(mA[hb] != mB[hb] || mn > m_o[hb])) {  // rare once the halves agree
          const float alpha = mn > m_o[hb] ? fast_exp2(m_o[hb] - mn) : 1.f;  // m_o = -inf -> 0
          m_o[hb] = mn;
          if (__ballot(alpha != 1.f)) {
#pragma unroll
            for (int c = 0; c < 4; ++c) o[4 * hb + c] *= alpha;
          }
          // P of the half whose reference is below m_o, brought to m_o
          const float fa = mA[hb] == mn ? 1.f : fast_exp2(mA[hb] - mn), fb = mB[hb] == mn ? 1.f : fast_exp2(mB[hb] - mn);
          if (__ballot(fa != 1.f)) pb[hb][0] = scale_bf16x8(pb[hb][0], fa);
          if (__ballot(fb != 1.f)) pb[hb][1] = scale_bf16x8(pb[hb][1], fb);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int hb = 0; hb < 2; ++hb) o[4 * hb + c] = mfma32(va[c][ks], pb[hb][ks], o[4 * hb + c]);
      if (it < ntiles) {
        __builtin_amdgcn_sched_barrier(0);
        read_v();
      }
    }
  }
  __syncthreads();  // the scorers' reference maxima and sums
  // accumulator layout: lane l, register r of block 4 hb + c holds dim 128 w4 + 32 c + 8 (r / 4) +
  // 4 (l / 32) + r % 4 of local head 32 hb + l % 32: in the list kernel head 32 hb + l % 32 of the
  // row, in the window kernel head 32 blockIdx.y + l % 32 of row 2 item + hb
  float mfin[2], lt[2];
#pragma unroll
  for (int hb = 0; hb < 2; ++hb) {
    // the two token halves' sums brought to the accumulators' reference (the larger final maximum)
    const int lh = 32 * hb + oj;
    const float ma = fin[2 * lh], la = fin[2 * lh + 1], mb = fin[2 * (64 + lh)], lb = fin[2 * (64 + lh) + 1];
    mfin[hb] = fmaxf(ma, mb);
    lt[hb] = (ma == mfin[hb] ? la : la * fast_exp2(ma - mfin[hb])) + (mb == mfin[hb] ? lb : lb * fast_exp2(mb - mfin[hb]));
  }
  // The normalised O of this wave (64 heads x 128 value columns, bf16) is staged head-major in the
  // tile buffers, idle since the barrier above (272 bytes per head: 256 + 16 of padding), and
  // written as 256-byte pieces of the head rows, four per store instruction: to the output, or
  // (SPLIT) to this split's partial, normalised by its own sum, which the merge weights back.
  uint8_t* ost = lds + w4 * (64 * 272);
#pragma unroll
  for (int hb = 0; hb < 2; ++hb) {
    const float inv = lt[hb] > 0.f ? 1.f / lt[hb] : 0.f;
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x16& ob = o[4 * hb + c];
        const u32x2 v = {pack_bf16x2(ob[4 * q] * inv, ob[4 * q + 1] * inv),
                         pack_bf16x2(ob[4 * q + 2] * inv, ob[4 * q + 3] * inv)};
        *reinterpret_cast<u32x2*>(ost + (32 * hb + oj) * 272 + (32 * c + 8 * q + 4 * (lane >> 5)) * 2) = v;
      }
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // (this wave's staging writes are done)
  // local head hh = 32 hb + h: head hh of the row, or (WIN) head 32 blockIdx.y + h of row 2 item + hb
  auto split_index = [&](int hb, int h, int64_t& pi) {
    const int64_t orow = WIN ? 2 * item + hb : row;
    pi = (orow * a.n_split + split) * 64 + (WIN ? 32 * (int)blockIdx.y : 32 * hb) + h;
    return orow < a.n_rows;  // WIN: the second row of an odd count is not written
  };
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int hh = 4 * k + (lane >> 4);
    const u32x4 v = *reinterpret_cast<const u32x4*>(ost + hh * 272 + 16 * (lane & 15));
    if (!SPLIT) {
      *reinterpret_cast<u32x4*>(a.out + (row * 64 + hh) * 512 + 128 * w4 + 8 * (lane & 15)) = v;
    } else {
      int64_t pi;
      if (split_index(hh >> 5, hh & 31, pi)) *reinterpret_cast<u32x4*>(a.part_o + pi * 512 + 128 * w4 + 8 * (lane & 15)) = v;
    }
  }
  if (w4 == 0 && lane < 32) {
#pragma unroll
    for (int hb = 0; hb < 2; ++hb) {
      if (!SPLIT) {
        if (a.lse) a.lse[row * 64 + 32 * hb + oj] = lt[hb] > 0.f ? (mfin[hb] + __log2f(lt[hb])) * kLn2 : -INFINITY;
      } else {
        int64_t pi;
        if (split_index(hb, oj, pi)) {
          a.part_ml[pi * 2] = mfin[hb];
          a.part_ml[pi * 2 + 1] = lt[hb];
        }
      }
    }
  }
}

// ============================================================================ MQA 16 x 128
// One wave per query row. K and V tiles (32 rows each) are staged through VGPRs into LDS;
// the configuration is small, so simplicity wins over the direct-load pipeline.
constexpr int kMqaKStride = 272;  // 256 + 16: K rows start 4 banks apart
constexpr int kMqaVStride = 288;  // 256 + 32: transposed V reads hit distinct banks

__global__ __launch_bounds__(64) void mqa_attn_kernel(AttnGeom a) {
  __shared__ __attribute__((aligned(16))) uint8_t lk[32 * kMqaKStride];
  __shared__ __attribute__((aligned(16))) uint8_t lv[32 * kMqaVStride];
  const int lane = threadIdx.x, g = lane >> 4, i16 = lane & 15, j = lane & 31;
  const int64_t row = xcd_band(blockIdx.x, a.n_rows);
  int cnt = a.count[row];
  cnt = cnt < 0 ? 0 : (cnt > a.k_cap ? a.k_cap : cnt);
  const int n = cnt, ntiles = (n + 31) / 32;
  const int32_t* slots = a.rows + row * a.k_cap;
  const u32x4* kg = reinterpret_cast<const u32x4*>(a.kv);
  const u32x4* vg = reinterpret_cast<const u32x4*>(a.v);

  // Q^T as the B operand: column = head i16, k-step s covers dims 32s + 8g .. +7
  u32x4 qb[4];
  {
    const u32x4* qp = reinterpret_cast<const u32x4*>(a.q + (row * 16 + i16) * 128 + 8 * g);
#pragma unroll
    for (int s = 0; s < 4; ++s) qb[s] = qp[4 * s];
  }
  f32x4 o[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) o[c] = f32x4{};
  float m = -INFINITY, l = 0.f;

  for (int it = 0; it < ntiles; ++it) {
    const int sl = it * 32 + j;
    int pr = sl < n ? slots[sl] : -1;
    pr = (pr >= 0 && (int64_t)pr < a.n_kv_rows) ? pr : -1;
    // stage K and V rows: 512 chunks of 16 bytes each, 8 per lane
    u32x4 kr[8], vr[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int u = k * 64 + lane, tok = u >> 4, ch = u & 15;
      const int r = __shfl(pr, tok);
      const int64_t base = (int64_t)(r >= 0 ? r : 0) * 16 + ch;
      kr[k] = kg[base];
      vr[k] = vg[base];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int u = k * 64 + lane, tok = u >> 4, ch = u & 15;
      *reinterpret_cast<u32x4*>(lk + tok * kMqaKStride + ch * 16) = kr[k];
      *reinterpret_cast<u32x4*>(lv + tok * kMqaVStride + ch * 16) = vr[k];
    }
    __syncthreads();
    const uint32_t vmask = (uint32_t)__ballot(pr >= 0);
    // ---- S^T = K Q^T, two 16-token M tiles; lane holds tokens 16mt + 4g + r of head i16
    f32x4 sacc[2] = {f32x4{}, f32x4{}};
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const u32x4 ka = *reinterpret_cast<const u32x4*>(lk + (16 * mt + i16) * kMqaKStride + (32 * s + 8 * g) * 2);
        sacc[mt] = mfma16(ka, qb[s], sacc[mt]);
      }
    float z[8];
    float mx = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int tk = 16 * mt + 4 * g + r;
        z[4 * mt + r] = ((vmask >> tk) & 1u) ? sacc[mt][r] * a.scale_log2 : -INFINITY;
        mx = fmaxf(mx, z[4 * mt + r]);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const bool need = mx > m + kLazy;
    if (__ballot(need)) {
      const float alpha = need ? fast_exp2(m - mx) : 1.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) o[c] *= alpha;
      l *= alpha;
      m = need ? mx : m;
    }
    float p[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      p[r] = z[r] == -INFINITY ? 0.f : fast_exp2(z[r] - m);
      l += p[r];
    }
    const u32x4 pb = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
    // ---- O^T += V^T P^T: k index 8g + v <-> token (v < 4 ? 4g + v : 16 + 4g + v - 4)
    const int vq = i16 >> 2, gq = i16 & 3;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const uint8_t* p0 = lv + (4 * g + vq) * kMqaVStride + (16 * c + 4 * gq) * 2;
      o[c] = mfma16(tr16_pair(p0, p0 + 16 * kMqaVStride), pb, o[c]);
    }
  }
  float lt = l + __shfl_xor(l, 16);
  lt += __shfl_xor(lt, 32);
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  uint16_t* orow = a.out + (row * 16 + i16) * 128 + 4 * g;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const u32x2 v = {pack_bf16x2(o[c][0] * inv, o[c][1] * inv), pack_bf16x2(o[c][2] * inv, o[c][3] * inv)};
    *reinterpret_cast<u32x2*>(orow + 16 * c) = v;
  }
  if (a.lse && g == 0) a.lse[row * 16 + i16] = lt > 0.f ? (m + __log2f(lt)) * kLn2 : -INFINITY;
}

// ============================================================================ split combine
// Log-sum-exp merge of the per-split partial results (the same rescaling the paper uses to
// merge partial attentions, Sec. 4.1.1 and App. B): each partial is stored in bf16, normalised by
// its own sum l_s, and weighted by l_s 2^(m_s - M) / sum_s l_s 2^(m_s - M). Grid (n_rows, H), block 128.
constexpr int kCombineRegs = 8;  // splits whose partials a thread holds at once
__global__ __launch_bounds__(128) void attn_combine_kernel(AttnGeom a, int H, int d_v) {
  const int64_t row = blockIdx.x;
  const int head = blockIdx.y;
  const int ns = a.n_split;
  auto pidx = [&](int s) { return (row * ns + s) * H + head; };
  if (ns <= kCombineRegs && d_v == 512) {
    // every split's maximum, sum and four values of this thread requested together (one round trip)
    const int d = (int)threadIdx.x * 4;
    float ms[kCombineRegs], ls[kCombineRegs];
    u32x2 pv[kCombineRegs];
#pragma unroll
    for (int s = 0; s < kCombineRegs; ++s) {
      ms[s] = -INFINITY;
      ls[s] = 0.f;
      pv[s] = u32x2{0u, 0u};
      if (s < ns) {
        const int64_t pi = pidx(s);
        ms[s] = a.part_ml[pi * 2];
        ls[s] = a.part_ml[pi * 2 + 1];
        pv[s] = *reinterpret_cast<const u32x2*>(a.part_o + pi * d_v + d);
      }
    }
    float M = -INFINITY;
#pragma unroll
    for (int s = 0; s < kCombineRegs; ++s) M = fmaxf(M, ms[s]);
    float L = 0.f;
    f32x4 acc = {};
#pragma unroll
    for (int s = 0; s < kCombineRegs; ++s) {
      if (!(ls[s] > 0.f)) continue;
      // the partial is normalised by its own sum ls: weight it back by ls 2^(m_s - M)
      const float wgt = ls[s] * fast_exp2(ms[s] - M);
      L += wgt;
      acc += wgt * f32x4{__uint_as_float(pv[s].x << 16), __uint_as_float(pv[s].x & 0xFFFF0000u),
                         __uint_as_float(pv[s].y << 16), __uint_as_float(pv[s].y & 0xFFFF0000u)};
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    const u32x2 v = {pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv)};
    *reinterpret_cast<u32x2*>(a.out + (row * H + head) * d_v + d) = v;
    if (a.lse && threadIdx.x == 0) a.lse[row * H + head] = L > 0.f ? (M + __log2f(L)) * kLn2 : -INFINITY;
    return;
  }
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, a.part_ml[pidx(s) * 2]);
  float L = 0.f;
  for (int s = 0; s < ns; ++s) {
    const int64_t pi = pidx(s);
    const float ms = a.part_ml[pi * 2], ls = a.part_ml[pi * 2 + 1];
    L += ls > 0.f ? ls * fast_exp2(ms - M) : 0.f;
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  for (int d = threadIdx.x * 4; d < d_v; d += 128 * 4) {
    f32x4 acc = {};
    for (int s = 0; s < ns; ++s) {
      const int64_t pi = pidx(s);
      const float ls = a.part_ml[pi * 2 + 1];
      if (!(ls > 0.f)) continue;
      // the partial is normalised by its own sum ls: weight it back by ls 2^(m_s - M)
      const float wgt = ls * fast_exp2(a.part_ml[pi * 2] - M);
      const u32x2 pv = *reinterpret_cast<const u32x2*>(a.part_o + pi * d_v + d);
      acc += wgt * f32x4{__uint_as_float(pv.x << 16), __uint_as_float(pv.x & 0xFFFF0000u),
                         __uint_as_float(pv.y << 16), __uint_as_float(pv.y & 0xFFFF0000u)};
    }
    const u32x2 v = {pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv)};
    *reinterpret_cast<u32x2*>(a.out + (row * H + head) * d_v + d) = v;
  }
  if (a.lse && threadIdx.x == 0) a.lse[row * H + head] = L > 0.f ? (M + __log2f(L)) * kLn2 : -INFINITY;
}

// ============================================================================ paged position -> cache row
__global__ __launch_bounds__(256) void translate_rows_kernel(const int32_t* __restrict__ idx, const int32_t* __restrict__ count,
                                                             int64_t n_rows, int k_cap, const int32_t* __restrict__ table,
                                                             int max_pages, int kv_page, int rows_per_seq, int64_t n_kv_rows,
                                                             int32_t* __restrict__ out) {
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= n_rows * k_cap) return;
  const int64_t row = id / k_cap;
  const int i = (int)(id - row * k_cap);
  int c = count[row];
  c = c < 0 ? 0 : (c > k_cap ? k_cap : c);
  int32_t r = -1;
  if (i < c) {
    const int32_t s = idx[id];
    const int64_t pg = s >= 0 ? s / kv_page : -1;
    if (pg >= 0 && pg < max_pages) {
      const int64_t ph = table[(row / rows_per_seq) * max_pages + pg];
      const int64_t cr = ph * kv_page + s % kv_page;
      if (ph >= 0 && cr < n_kv_rows) r = (int32_t)cr;
    }
  }
  out[id] = r;
}

// ============================================================================ host launchers
template <bool SPLIT>
static void launch_mla_kernel(dim3 grid, const AttnGeom& a, hipStream_t st) {
  hipLaunchKernelGGL((mla_attn_kernel<SPLIT>), grid, dim3(512), 0, st, a);
}

hipError_t launch_mla_attn(const AttnGeom& a, hipStream_t st) {
  if (a.n_rows == 0) return hipSuccess;
  if (a.n_split > 1) {
    launch_mla_kernel<true>(dim3((unsigned)a.n_rows, (unsigned)a.n_split), a, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_attn_combine(a, 64, 512, st);
  }
  launch_mla_kernel<false>(dim3((unsigned)a.n_rows), a, st);
  return hipGetLastError();
}

hipError_t launch_mla_attn_part(const AttnGeom& a, hipStream_t st) {
  if (a.n_rows == 0) return hipSuccess;
  launch_mla_kernel<true>(dim3((unsigned)a.n_rows), a, st);
  return hipGetLastError();
}

hipError_t launch_mla_attn_window(const AttnGeom& a, hipStream_t st) {
  if (a.n_rows == 0) return hipSuccess;
  hipLaunchKernelGGL((mla_attn_kernel<true, true>), dim3((unsigned)((a.n_rows + 1) / 2), 2u), dim3(512), 0,
                     st, a);
  return hipGetLastError();
}

hipError_t launch_mqa_attn(const AttnGeom& a, hipStream_t st) {
  if (a.n_rows == 0) return hipSuccess;
  hipLaunchKernelGGL(mqa_attn_kernel, dim3((unsigned)a.n_rows), dim3(64), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_attn_combine(const AttnGeom& a, int H, int d_v, hipStream_t st) {
  hipLaunchKernelGGL(attn_combine_kernel, dim3((unsigned)a.n_rows, (unsigned)H), dim3(128), 0, st, a, H, d_v);
  return hipGetLastError();
}

hipError_t launch_translate_rows(const int32_t* idx, const int32_t* count, int64_t n_rows, int k_cap,
                                 const int32_t* page_table, int max_pages, int kv_page, int rows_per_seq,
                                 int64_t n_kv_rows, int32_t* out_rows, hipStream_t st) {
  const int64_t n = n_rows * k_cap;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(translate_rows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, idx, count, n_rows, k_cap,
                     page_table, max_pages, kv_page, rows_per_seq, n_kv_rows, out_rows);
  return hipGetLastError();
}

}  // namespace lsa
