// LSA indexer kernels for gfx950: mean-key cache, coarse page scoring, page top-M,
// fine token scoring, token top-K with the streaming merge, and run encoding.
//
// Paper: "LongCat Sparse Attention" (arXiv 2608.01662), Sec. 2.2 Eq. (1)-(2),
// Sec. 3.1 Eq. (6)-(7), Sec. 3.3 Eq. (9)-(12).
//
// Score layout. Both scoring stages are dense contractions Q_I (heads x d_I) times keys
// (d_I x 32 keys) on v_mfma_f32_32x32x16_bf16: the 32 MFMA rows are the indexer heads (zero-
// padded when H_I < 32), the 32 columns are keys. In the accumulator layout each lane owns one
// key column and 16 heads, so ReLU, the head weights and the sum over heads (Eq. 1 / Eq. 9) are
// 16 in-lane FMAs plus one exchange with the lane 32 apart. fp8 keys are widened to bf16 exactly
// (e4m3 has 4 significant bits) and the per-token scale is applied after the sum, which is
// exact algebra since ReLU(s x) = s ReLU(x) for s > 0.
//
// The contraction over d_I uses a permuted order of the dimensions: in k-step s the lanes of
// half h supply dims (d_I/2)*h + 8*s .. +7 of both operands. Any permutation applied to both
// operands leaves the dot product unchanged, and this one lets every lane read one contiguous
// run of key bytes.
#include <atomic>

#include "device.hpp"
#include "launch.hpp"

namespace lsa {

// 8 e4m3fn codes (two dwords) -> one bf16x8 MFMA operand with gfx950's packed converter: two
// codes per instruction (scale 1.0, so the exact values come out as bf16).
__device__ __forceinline__ u32x4 fp8x8_to_bf16x8_pk(uint32_t a, uint32_t b) {
  return u32x4{__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(a, 1.0f, false)),
               __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(a, 1.0f, true)),
               __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(b, 1.0f, false)),
               __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(b, 1.0f, true))};
}

// ============================================================================ row geometry
struct RowInfo {
  int64_t t;       // query position
  int valid;       // 0: skip the row (bad context length)
  int64_t lo, hi;  // eligible range E_t = [lo, hi] (empty if lo > hi)
  int64_t p_lo, p_hi;
};

__device__ __forceinline__ RowInfo row_info(const IndexGeom& g, int64_t row) {
  RowInfo r;
  if (g.ctx_len) {
    const int64_t c = g.ctx_len[row];
    r.valid = (c >= 1 && c <= (int64_t)g.max_pages * g.kv_page);
    r.t = r.valid ? c - 1 : 0;
  } else {
    r.valid = 1;
    r.t = g.q_start + row;
  }
  r.lo = g.k_sink;
  r.hi = r.t - g.k_swa;
  r.p_lo = r.lo / g.P;
  r.p_hi = r.hi >= r.lo ? r.hi / g.P : r.p_lo - 1;
  return r;
}

// Physical page of logical page `p` of sequence `seq` (-1 if the entry is out of range).
__device__ __forceinline__ int64_t phys_page(const IndexGeom& g, int64_t seq, int64_t p) {
  if (p < 0 || p >= g.max_pages) return -1;
  const int64_t ph = g.page_table[seq * g.max_pages + p];
  return (ph >= 0 && ph < g.n_phys) ? ph : -1;
}

// ============================================================================ block cache (Stage 1)
// Sub-block handled by work item `item`: item itself (whole cache), or the sub-block holding token
// rows[item] (incremental update); -1 when that row is out of range or in the incomplete tail.
__device__ __forceinline__ int64_t block_of_item(int64_t item, const int64_t* __restrict__ rows, int64_t n_tok, int B) {
  if (rows == nullptr) return item;
  const int64_t r = rows[item];
  return (r >= 0 && r < n_tok && r / B < n_tok / B) ? r / B : -1;
}

// Mean keys (Eq. 9). One thread per (work item, group of 4 dims): fp32 sum of s_i * k_i over the
// B tokens, one multiply by 1/B (B is a power of two, exact), one round-to-nearest-even to bf16.
template <bool FP8>
__global__ __launch_bounds__(256) void block_means_kernel(int64_t n_items, const int64_t* __restrict__ rows, int64_t n_tok,
                                                          int D, int B, const void* __restrict__ k,
                                                          const float* __restrict__ ks, uint16_t* __restrict__ out) {
  const int groups = D / 4;
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= n_items * groups) return;
  const int64_t item = id / groups;
  const int gq = (int)(id - item * groups);
  const int64_t sub = block_of_item(item, rows, n_tok, B);
  if (sub < 0) return;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < B; ++i) {
    const int64_t tok = sub * B + i;
    if (FP8) {
      const uint32_t v = reinterpret_cast<const uint32_t*>(k)[tok * groups + gq];
      const f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8(v, false);
      const f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8(v, true);
      const float s = ks[tok];
      acc[0] += s * lo.x; acc[1] += s * lo.y; acc[2] += s * hi.x; acc[3] += s * hi.y;
    } else {
      const u32x2 v = reinterpret_cast<const u32x2*>(k)[tok * groups + gq];
      acc[0] += __uint_as_float(v.x << 16); acc[1] += __uint_as_float(v.x & 0xFFFF0000u);
      acc[2] += __uint_as_float(v.y << 16); acc[3] += __uint_as_float(v.y & 0xFFFF0000u);
    }
  }
  const float inv = 1.0f / (float)B;
  u32x2 o;
  o.x = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  o.y = pack_bf16x2(acc[2] * inv, acc[3] * inv);
  reinterpret_cast<u32x2*>(out)[sub * groups + gq] = o;
}

// bf16 bits of x rounded to nearest, ties to even, in one step from fp64: the float rounded
// toward zero keeps x's leading 24 bits exactly, and whether anything non-zero lies below them
// only matters as a sticky bit (finite values within the float range).
__device__ __forceinline__ uint32_t bf16_rne_from_f64(double x) {
  const float t = __double2float_rz(x);
  const uint32_t b = __float_as_uint(t);
  const bool below = (double)t != x;
  const uint32_t lsb = (b >> 16) & 1u, half = (b >> 15) & 1u;
  const bool rest = (b & 0x7FFFu) != 0u || below;
  return (b >> 16) + (half & (uint32_t)(rest || lsb));
}

// Min-max extrema (Eq. 13). One thread per (work item, group of 4 dims): each dequantised key
// s_i * k_i is formed exactly in fp64 (24-bit scale times 4-bit code), the extrema are exact, and
// each is rounded once to bf16. Output row: [k_max (D) | k_min (D)].
template <bool FP8>
__global__ __launch_bounds__(256) void block_minmax_kernel(int64_t n_items, const int64_t* __restrict__ rows, int64_t n_tok,
                                                           int D, int B, const void* __restrict__ k,
                                                           const float* __restrict__ ks, uint16_t* __restrict__ out) {
  const int groups = D / 4;
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= n_items * groups) return;
  const int64_t item = id / groups;
  const int gq = (int)(id - item * groups);
  const int64_t sub = block_of_item(item, rows, n_tok, B);
  if (sub < 0) return;
  double mx[4], mn[4];
  for (int i = 0; i < B; ++i) {
    const int64_t tok = sub * B + i;
    double v[4];
    if (FP8) {
      const uint32_t c = reinterpret_cast<const uint32_t*>(k)[tok * groups + gq];
      const f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8(c, false);  // codes decode exactly
      const f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8(c, true);
      const double s = (double)ks[tok];
      v[0] = s * (double)lo.x; v[1] = s * (double)lo.y; v[2] = s * (double)hi.x; v[3] = s * (double)hi.y;
    } else {
      const u32x2 c = reinterpret_cast<const u32x2*>(k)[tok * groups + gq];
      v[0] = (double)__uint_as_float(c.x << 16); v[1] = (double)__uint_as_float(c.x & 0xFFFF0000u);
      v[2] = (double)__uint_as_float(c.y << 16); v[3] = (double)__uint_as_float(c.y & 0xFFFF0000u);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      mx[e] = (i == 0 || v[e] > mx[e]) ? v[e] : mx[e];
      mn[e] = (i == 0 || v[e] < mn[e]) ? v[e] : mn[e];
    }
  }
  u32x2 hi, lo;
  hi.x = bf16_rne_from_f64(mx[0]) | (bf16_rne_from_f64(mx[1]) << 16);
  hi.y = bf16_rne_from_f64(mx[2]) | (bf16_rne_from_f64(mx[3]) << 16);
  lo.x = bf16_rne_from_f64(mn[0]) | (bf16_rne_from_f64(mn[1]) << 16);
  lo.y = bf16_rne_from_f64(mn[2]) | (bf16_rne_from_f64(mn[3]) << 16);
  u32x2* row = reinterpret_cast<u32x2*>(out + sub * 2 * D);
  row[gq] = hi;
  row[groups + gq] = lo;
}

// ============================================================================ operand loads
// A operand: 32 (padded) heads of one query row. Lane (head j, half h), k-step s: 8 bf16 at
// dims (D/2)*h + 8*s.
template <int D>
__device__ __forceinline__ void load_query_operand(const uint16_t* __restrict__ q, int H, int64_t row, int lane,
                                                   u32x4 (&a)[D / 16]) {
  const int j = lane & 31, h = lane >> 5;
  if (j < H) {
    const uint16_t* p = q + (row * H + j) * D + (D / 2) * h;
#pragma unroll
    for (int s = 0; s < D / 16; ++s) a[s] = *reinterpret_cast<const u32x4*>(p + 8 * s);
  } else {
#pragma unroll
    for (int s = 0; s < D / 16; ++s) a[s] = u32x4{0, 0, 0, 0};
  }
}

// Head weights of the 16 heads this lane holds in the accumulator: 8*(r/4) + 4*h + r%4.
__device__ __forceinline__ void load_head_weights(const float* __restrict__ w, int H, int64_t row, int lane, float (&wr)[16]) {
  const int h = lane >> 5;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int head = 8 * (r / 4) + 4 * h + (r % 4);
    wr[r] = head < H ? w[row * H + head] : 0.f;
  }
}

// B operand for one key row: lane half h reads dims [(D/2)*h, (D/2)*h + D/2) of key `krow`.
template <int D, bool FP8>
__device__ __forceinline__ void load_key_operand(const void* __restrict__ k, int64_t krow, int lane, u32x4 (&b)[D / 16]) {
  const int h = lane >> 5;
  if (FP8) {
    const u32x4* p = reinterpret_cast<const u32x4*>(reinterpret_cast<const uint8_t*>(k) + krow * D + (D / 2) * h);
#pragma unroll
    for (int v = 0; v < D / 32; ++v) {
      const u32x4 raw = p[v];  // 16 codes = k-steps 2v, 2v+1
      b[2 * v] = fp8x8_to_bf16x8(raw.x, raw.y);
      b[2 * v + 1] = fp8x8_to_bf16x8(raw.z, raw.w);
    }
  } else {
    const u32x4* p = reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(k) + krow * D + (D / 2) * h);
#pragma unroll
    for (int s = 0; s < D / 16; ++s) b[s] = p[s];
  }
}

// max(x, 0) as one integer max on the bit pattern: negative floats (sign bit set) are negative
// integers and become +0, non-negative floats are unchanged. fmaxf would first quiet signalling
// NaNs with an extra v_max x, x, since an MFMA result is not known to be canonical.
__device__ __forceinline__ float relu(float x) { return __int_as_float(max(__float_as_int(x), 0)); }

// sum_j w_j ReLU(acc_j) over the 32 heads of this lane's key column (Eq. 1 / Eq. 9), as four
// interleaved partial sums (a fixed order, so every tile and row rounds the same way). The two
// lane halves hold 16 heads each; v_permlane32_swap hands each lane its partner's half sum
// (a VALU exchange, no LDS round trip), and a + b == b + a, so both lanes agree bit for bit.
__device__ __forceinline__ float head_reduce(const f32x16& acc, const float (&wr)[16]) {
  float p[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int r = 0; r < 16; ++r) p[r & 3] = fmaf(wr[r], relu(acc[r]), p[r & 3]);
  const float v = (p[0] + p[1]) + (p[2] + p[3]);
  const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(x[0]) + __uint_as_float(x[1]);
}

// A operand of min-max pooling (Eq. 13): per dimension max(q k_max, q k_min) = q+ k_max + q- k_min
// with q+ = max(q, 0), q- = min(q, 0), so the block score is one dot product of width 2D between
// [q+ | q-] and the cached [k_max | k_min]. Lane half 0 holds q+, half 1 holds q-; k-step s covers
// dims 8s..8s+7 in both halves (the key operand's halves are k_max and k_min of the same dims).
template <int D>
__device__ __forceinline__ void load_query_minmax(const uint16_t* __restrict__ q, int H, int64_t row, int lane,
                                                  u32x4 (&a)[D / 8]) {
  const int j = lane & 31, h = lane >> 5;
  // per bf16 half-word: all ones where the value is negative (sign bit set)
  auto neg = [](uint32_t v) { return ((v >> 15) & 0x00010001u) * 0xFFFFu; };
  auto part = [&](uint32_t v) { return h ? (v & neg(v)) : (v & ~neg(v)); };
#pragma unroll
  for (int s = 0; s < D / 8; ++s) {
    if (j < H) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(q + (row * H + j) * D + 8 * s);
      a[s] = u32x4{part(v.x), part(v.y), part(v.z), part(v.w)};
    } else {
      a[s] = u32x4{0, 0, 0, 0};
    }
  }
}

// fp8 keys are scored on the fp8 matrix cores (Eq. 1 / Eq. 11 with e4m3 key codes as they are
// stored). The bf16 query of each head is scaled by a power of two 2^E (its largest |q| lands in
// [2^7, 2^8)) and split into two e4m3 terms, q 2^E = hi + lo: the hi term keeps the leading 4
// significant bits (round to nearest even), the lo term the remaining ones, so the split is exact
// for every element of at least 2^-2 after scaling, i.e. within 2^10 of the head's largest;
// smaller ones are off by at most half the e4m3 subnormal step, 2^-10 after scaling, 2^-18 of the
// head's largest element. The factor 2^-E goes into the head weight: w ReLU(x) = (w 2^-E) ReLU(x 2^E).
// Operand i of a lane holds dims (D/2) h + 32 i .. + 31, the order the key bytes have in LDS.
__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }

// four bf16 values (two dwords) times sc -> the e4m3 codes of their hi and lo terms (one dword each)
__device__ __forceinline__ void split_fp8x4(uint32_t w0, uint32_t w1, float sc, uint32_t& hi, uint32_t& lo) {
  const float x0 = bf16_lo(w0) * sc, x1 = bf16_hi(w0) * sc, x2 = bf16_lo(w1) * sc, x3 = bf16_hi(w1) * sc;
  int h = __builtin_amdgcn_cvt_pk_fp8_f32(x0, x1, 0, false);
  h = __builtin_amdgcn_cvt_pk_fp8_f32(x2, x3, h, true);
  const f32x2 b01 = __builtin_amdgcn_cvt_pk_f32_fp8(h, false), b23 = __builtin_amdgcn_cvt_pk_f32_fp8(h, true);
  int l = __builtin_amdgcn_cvt_pk_fp8_f32(x0 - b01.x, x1 - b01.y, 0, false);  // exact differences
  l = __builtin_amdgcn_cvt_pk_fp8_f32(x2 - b23.x, x3 - b23.y, l, true);
  hi = (uint32_t)h;
  lo = (uint32_t)l;
}

// From the bf16 query operand a (as load_query_operand holds it) and the head weights wr (as
// load_head_weights holds them): the fp8 operands qh, ql of the D/64 products per tile, and wr
// multiplied by 2^-E of each head.
template <int D>
__device__ __forceinline__ void query_fp8(const u32x4 (&a)[D / 16], int lane, i32x8 (&qh)[D / 64],
                                          i32x8 (&ql)[D / 64], float (&wr)[16]) {
  // largest |q| of this lane's head (its D/2 dims here, the other half in lane ^ 32)
  uint32_t mx = 0;  // bf16 magnitudes order like their bit patterns
  auto mag2 = [](uint32_t d) { return max(d & 0x7FFFu, (d >> 16) & 0x7FFFu); };
#pragma unroll
  for (int s = 0; s < D / 16; ++s) {
    const u32x4 v = a[s];
    mx = max(mx, max(max(mag2(v.x), mag2(v.y)), max(mag2(v.z), mag2(v.w))));
  }
  mx = max(mx, (uint32_t)__shfl_xor((int)mx, 32));
  const int ex = (int)((mx >> 7) & 0xFF) - 127;  // floor(log2 max|q|) for a normal maximum
  int E = mx == 0u ? 0 : 7 - ex;
  E = E < -60 ? -60 : (E > 60 ? 60 : E);
  const float sc = __uint_as_float((uint32_t)(E + 127) << 23);
#pragma unroll
  for (int i = 0; i < D / 64; ++i) {
    uint32_t h[8], l[8];
#pragma unroll
    for (int u = 0; u < 4; ++u) {  // a[4i + u] holds dims (D/2) h + 32 i + 8 u .. + 7
      const u32x4 v = a[4 * i + u];
      split_fp8x4(v.x, v.y, sc, h[2 * u], l[2 * u]);
      split_fp8x4(v.z, v.w, sc, h[2 * u + 1], l[2 * u + 1]);
    }
    qh[i] = i32x8{(int)h[0], (int)h[1], (int)h[2], (int)h[3], (int)h[4], (int)h[5], (int)h[6], (int)h[7]};
    ql[i] = i32x8{(int)l[0], (int)l[1], (int)l[2], (int)l[3], (int)l[4], (int)l[5], (int)l[6], (int)l[7]};
  }
  // head of accumulator register r: 8 (r / 4) + 4 h + r % 4; lane `head` holds that head's exponent
  const int hh = lane >> 5;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int Er = __shfl(E, 8 * (r / 4) + 4 * hh + (r % 4));
    wr[r] *= __uint_as_float((uint32_t)(127 - Er) << 23);
  }
}

// One direct global->LDS load (16 or 4 bytes per lane; lane i writes LDS bytes [lds + SIZE*i, ..)),
// issued from asm so that the compiler's wait insertion does not drain it before LDS reads that it
// cannot prove disjoint; callers wait with an explicit vmcnt. M0 (the load's LDS base) is saved and
// restored; the s_nop is the wait state between writing M0 and the load reading it.
// The address is a wave-uniform 64-bit base plus a per-lane 32-bit byte offset.
template <int SIZE>
__device__ __forceinline__ void lds_dma(const void* base, uint32_t off, uint32_t lds) {
  static_assert(SIZE == 16 || SIZE == 4, "load size");
  uint32_t save;
  if constexpr (SIZE == 16)
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2\n\ts_mov_b32 m0, %0"
                 : "=&s"(save) : "v"(off), "s"(base), "s"(lds) : "memory");
  else
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %3\n\ts_nop 0\n\tglobal_load_lds_dword %1, %2\n\ts_mov_b32 m0, %0"
                 : "=&s"(save) : "v"(off), "s"(base), "s"(lds) : "memory");
}
// Every LDS read this wave issued has returned its data.
__device__ __forceinline__ void lds_read_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// ============================================================================ Stage 1: coarse page scores
// Eq. (9), or Eq. (13) with MINMAX. Grid: (ceil(n_rows / R), chunks). Each wave takes tiles of 32
// block keys of the chunk; R query rows share each loaded tile (prefill). Output: order keys of
// the page scores, page_keys[row * ld + p] for eligible pages p.
// STAGED (prefill mean keys, rows of at most kCoarseStagedTiles tiles; the tile's 32 block keys are
// consecutive rows of the cache): one wave per workgroup takes every tile of its R rows, the rows
// with the most eligible pages first so that the long workgroups do not form the tail of the
// launch; it copies its next tile into its own LDS buffer by direct loads while it scores the
// current one, whole key rows per 16 (or 8) consecutive lanes, so that a load touches 4 (or 8)
// rows instead of one row per lane; granule c of row t sits at slot c ^ coarse_swz(t) of the row,
// which keeps the operand reads (16 rows, one granule) free of bank conflicts. Otherwise four waves
// share the tiles of R rows and read the keys straight into the operand layout (long rows: the
// block keys no longer fit the L2, and four rows per tile read them fewer times).
constexpr int kCoarseRowsStaged = 3;   // query rows of a staged workgroup (register budget)
constexpr int kCoarseStagedTiles = 64; // longest row (in 32-key tiles) taken by the staged kernel
template <int GR>  // 16-byte granules per key row: 16 (d = 128) or 8 (d = 64)
__device__ __forceinline__ int coarse_swz(int t) { return GR == 16 ? (t & 15) : ((t >> 1) & 7); }

template <int D, int R, bool PAGED, bool MINMAX, bool STAGED = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void coarse_kernel(IndexGeom g, int64_t n_rows, const uint16_t* __restrict__ q,
                                                     const float* __restrict__ w, const uint16_t* __restrict__ kmean,
                                                     uint32_t* __restrict__ page_keys, int64_t ld, int tiles_per_chunk) {
  constexpr int DK = MINMAX ? 2 * D : D;  // width of a block key and of the dot product
  constexpr int KS = DK / 16;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, j = lane & 31;
  static_assert(!STAGED || (!PAGED && !MINMAX), "staged tiles are consecutive mean keys");
  const int64_t row0 = (int64_t)(STAGED ? gridDim.x - 1 - blockIdx.x : blockIdx.x) * R;
  const int nsub = g.P / g.B;

  if constexpr (PAGED) {
    // Decode: one row, chunks of 8 tiles, wave wv scoring tiles wv and wv + 4 of its chunk. The
    // page-table entries of both tiles and the query are requested before the context length is
    // known (any page below max_pages lies inside the sequence's table row), and both tiles' block
    // keys together, so the scores wait for two round trips instead of four. Pages past the
    // row's eligible range are scored but not stored.
    static_assert(R == 1 && !STAGED, "paged scoring takes one row per workgroup");
    const int64_t row = row0, p_base = g.k_sink / g.P;  // first eligible page (k_sink only)
    const int64_t tile_beg = (int64_t)blockIdx.y * tiles_per_chunk;
    int64_t pp[2], ph[2];
    int sub[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t sb = (tile_beg + wv + 4 * u) * 32 + j;  // sub-block counted from the first eligible page
      pp[u] = p_base + sb / nsub;
      sub[u] = (int)(sb % nsub);
      ph[u] = phys_page(g, row, pp[u]);
    }
    u32x4 a[KS];
    float wr[16];
    if constexpr (MINMAX) load_query_minmax<D>(q, g.H, row, lane, a);
    else load_query_operand<D>(q, g.H, row, lane, a);
    load_head_weights(w, g.H, row, lane, wr);
    const RowInfo ri = row_info(g, row);
    if (!ri.valid || ri.p_hi < ri.p_lo) return;
    const int64_t n_tiles = ((ri.p_hi - ri.p_lo + 1) * nsub + 31) / 32;
    u32x4 b[2][KS];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t mrow = ph[u] >= 0 ? ph[u] * nsub + sub[u] : 0;
      const u32x4* pk = reinterpret_cast<const u32x4*>(kmean + mrow * DK + (DK / 2) * (lane >> 5));
#pragma unroll
      for (int s = 0; s < KS; ++s) b[u][s] = pk[s];
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t tile = tile_beg + wv + 4 * u;
      if (4 * u + wv >= tiles_per_chunk || tile >= n_tiles) break;  // (wave-uniform)
      f32x16 acc = {};
#pragma unroll
      for (int s = 0; s < KS; ++s) acc = mfma32(a[s], b[u][s], acc);
      float v = head_reduce(acc, wr);
      for (int o = 1; o < nsub; o <<= 1) v += __shfl_xor(v, o);  // sum the sub-blocks of a page
      if (lane < 32 && sub[u] == 0 && pp[u] <= ri.p_hi) page_keys[row * ld + pp[u]] = ph[u] >= 0 ? score_key(v) : 0u;
    }
    return;
  }

  RowInfo ri[R];
  int64_t max_tiles = 0;
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row0 + r;
    ri[r] = row < n_rows ? row_info(g, row) : RowInfo{0, 0, 1, 0, 0, -1};
    if (ri[r].valid && ri[r].p_hi >= ri[r].p_lo) {
      const int64_t nt = ((ri[r].p_hi - ri[r].p_lo + 1) * nsub + 31) / 32;
      max_tiles = nt > max_tiles ? nt : max_tiles;
    }
  }
  const int64_t tile_beg = (int64_t)blockIdx.y * tiles_per_chunk;
  const int64_t tile_end = tile_beg + tiles_per_chunk < max_tiles ? tile_beg + tiles_per_chunk : max_tiles;
  if (tile_beg >= tile_end) return;

  u32x4 a[R][KS];
  float wr[R][16];
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const int64_t row = row0 + r < n_rows ? row0 + r : n_rows - 1;
    if constexpr (MINMAX) load_query_minmax<D>(q, g.H, row, lane, a[r]);
    else load_query_operand<D>(q, g.H, row, lane, a[r]);
    load_head_weights(w, g.H, row, lane, wr[r]);
  }
  const int64_t p_base = ri[0].p_lo;  // identical for every row (depends on k_sink only)

  if constexpr (STAGED) {  // (the launcher checks 0 < n_sub and n_sub * row bytes < 2^32)
    constexpr int RB = DK * 2, GR = RB / 16;  // key row bytes, granules
    constexpr int NDMA = 32 * RB / 1024;      // direct loads per tile (1 KB each)
    constexpr int RPL = 1024 / RB;            // key rows per load
    __shared__ __attribute__((aligned(16))) uint8_t csm[2][32 * RB];
    const int64_t row_lim = g.n_sub - 1;      // (rows past the cache are loaded clamped, scored as 0)
    // load slot: lane -> key row RPL m + lane / GR of the tile, granule (lane % GR) ^ swz(row)
    const int tl = lane / GR, cl = lane % GR;
    const uint8_t* base = reinterpret_cast<const uint8_t*>(kmean);  // byte offsets fit 32 bits (host check)
    auto issue = [&](int64_t tile, int buf) {
      const int64_t r0 = p_base * nsub + tile * 32;
      const uint32_t lds = lds_addr(&csm[buf][0]);
#pragma unroll
      for (int m = 0; m < NDMA; ++m) {
        const int t = RPL * m + tl;
        const int64_t rr = r0 + t < row_lim ? r0 + t : row_lim;
        const uint32_t off = (uint32_t)(rr * RB + 16 * (cl ^ coarse_swz<GR>(t)));
        lds_dma<16>(base, off, lds + 1024 * m);
      }
    };
    // operand read: lane (j, h) at k-step s takes granule (GR / 2) h + s of key row j
    const uint32_t rd = (uint32_t)(j * RB);
    const int swz_j = coarse_swz<GR>(j), h = lane >> 5;
    int buf = 0;
    issue(tile_beg, 0);
    for (int64_t tile = tile_beg; tile < tile_end; ++tile) {
      const bool more = tile + 1 < tile_end;
      if (more) issue(tile + 1, buf ^ 1);
      if (more) vm_wait<NDMA>();  // this tile's loads (and earlier stores) are done
      else vm_wait<0>();
      const uint8_t* tb = &csm[buf][0];
      u32x4 b[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s)
        b[s] = *reinterpret_cast<const u32x4*>(tb + rd + 16 * ((((GR / 2) * h) + s) ^ swz_j));
      const int64_t sb = tile * 32 + j;
      const int64_t p = p_base + sb / nsub;
      const int sub_in_page = (int)(sb % nsub);
      const bool okp = p * nsub + sub_in_page < g.n_sub;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        f32x16 acc = {};
#pragma unroll
        for (int s = 0; s < KS; ++s) acc = mfma32(a[r][s], b[s], acc);
        float v = head_reduce(acc, wr[r]);
        for (int o = 1; o < nsub; o <<= 1) v += __shfl_xor(v, o);  // sum the sub-blocks of a page
        const int64_t row = row0 + r;
        if (lane < 32 && sub_in_page == 0 && row < n_rows && ri[r].valid && p <= ri[r].p_hi)
          page_keys[row * ld + p] = okp ? score_key(v) : 0u;
      }
      lds_read_wait();  // the operand reads of this buffer are done before it is refilled
      buf ^= 1;
    }
    return;
  }

  for (int64_t tile = tile_beg + wv; tile < tile_end; tile += 4) {
    const int64_t sb = tile * 32 + j;            // sub-block counted from the first eligible page
    const int64_t p = p_base + sb / nsub;
    const int sub_in_page = (int)(sb % nsub);
    int64_t mrow = 0;
    bool okp = true;
    okp = p * nsub + sub_in_page < g.n_sub;
    mrow = okp ? p * nsub + sub_in_page : 0;
    u32x4 b[KS];
    {
      const u32x4* pk = reinterpret_cast<const u32x4*>(kmean + mrow * DK + (DK / 2) * (lane >> 5));
#pragma unroll
      for (int s = 0; s < KS; ++s) b[s] = pk[s];
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      f32x16 acc = {};
#pragma unroll
      for (int s = 0; s < KS; ++s) acc = mfma32(a[r][s], b[s], acc);
      float v = head_reduce(acc, wr[r]);
      for (int o = 1; o < nsub; o <<= 1) v += __shfl_xor(v, o);  // sum the sub-blocks of a page
      const int64_t row = row0 + r;
      if (lane < 32 && sub_in_page == 0 && row < n_rows && ri[r].valid && p <= ri[r].p_hi)
        page_keys[row * ld + p] = okp ? score_key(v) : 0u;
    }
  }
}

// ============================================================================ block-wide top-k
// Threshold T and tie count of the k largest keys among keys[0..n) (LDS or global memory), by at
// most four 8-bit radix passes: the selection is {i : key_i > T} plus the first `take_eq` indices
// with key_i == T. (1 <= k <= n.)
// hist[0..256) must be zero on entry (cleared before a barrier) and is zero again on return: the
// scanning wave clears the bins as it reads them, before the barrier that publishes the boundary
// bin. Two block barriers per pass. The boundary bin is published in the function's own LDS slots,
// which a pass rewrites only after its counting barrier, when every wave has read the previous
// pass's, so no barrier guards the reads and the caller may reuse its LDS right away. When the
// boundary bin is taken whole (its count equals the rank still missing) and is not the bin of key
// 0, the search stops there: T is the largest key below the bin and take_eq is 0, which selects
// exactly the same set (every key equal to the exact threshold lies in that bin and is taken).
// That needs every candidate key that shares the bin's digits to be among keys[0..n): when keys
// holds only the candidates that share their top 11 bits, the stop is allowed from the second
// pass on (first_exit = 1), whose bins fix 16 bits.
template <int NT>
__device__ void radix_threshold(const uint32_t* keys, int n, int k, uint32_t* hist, uint32_t& T, int& take_eq,
                                int first_exit = 0) {
  __shared__ int slot[3];  // boundary bin, keys in the bins above it, keys in it
  uint32_t prefix = 0, mask = 0;
  int rem = k;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int i = threadIdx.x; i < n; i += NT) {
      const uint32_t key = keys[i];
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      const int l = threadIdx.x;
      const uint32_t c[4] = {hist[4 * l], hist[4 * l + 1], hist[4 * l + 2], hist[4 * l + 3]};
#pragma unroll
      for (int bq = 0; bq < 4; ++bq) hist[4 * l + bq] = 0;  // cleared for the next pass
      const uint32_t tot = c[0] + c[1] + c[2] + c[3];
      uint32_t suf = tot;  // sum of totals of lanes >= l
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t x = __shfl_down(suf, o);
        if (l + o < 64) suf += x;
      }
      uint32_t ge = suf - tot;  // keys in bins above this lane's four
      for (int bq = 3; bq >= 0; --bq) {
        const uint32_t above = ge;
        ge += c[bq];
        if (above < (uint32_t)rem && ge >= (uint32_t)rem) {
          slot[0] = 4 * l + bq;
          slot[1] = (int)above;
          slot[2] = (int)c[bq];
        }
      }
    }
    __syncthreads();
    const uint32_t d = (uint32_t)slot[0];
    rem -= slot[1];
    prefix |= d << shift;
    mask |= 0xFFu << shift;
    if (pass >= first_exit && pass < 3 && slot[2] == rem && prefix != 0u) {  // (uniform) the bin is taken whole
      T = prefix - 1u;
      take_eq = 0;
      return;
    }
  }
  T = prefix;
  take_eq = rem;
}

// Visits, in index order, every selected index of keys[0..n) (key > T, or key == T among the
// first take_eq such) and calls emit(rank, i). Returns the number selected. The caller writes
// wsum[0..2 NT/64) again only after a barrier.
template <int NT, typename F>
__device__ int select_compact(const uint32_t* keys, int n, uint32_t T, int take_eq, int* wsum, F&& emit) {
  constexpr int NW = NT / 64;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int base_eq = 0, base_out = 0;
  for (int c = 0; c < n; c += NT) {
    const int i = c + threadIdx.x;
    const uint32_t key = i < n ? keys[i] : 0u;
    const bool eq = i < n && key == T;
    const uint64_t beq = __ballot(eq);
    if (lane == 0) wsum[wv] = __popcll(beq);
    __syncthreads();
    int eq_prefix = 0, eq_total = 0;
#pragma unroll
    for (int x = 0; x < NW; ++x) {
      const int v = wsum[x];
      eq_prefix += x < wv ? v : 0;
      eq_total += v;
    }
    const int eq_rank = base_eq + eq_prefix + __popcll(beq & lanemask_lt());
    const bool sel = i < n && (key > T || (eq && eq_rank < take_eq));
    const uint64_t bsel = __ballot(sel);
    if (lane == 0) wsum[NW + wv] = __popcll(bsel);
    __syncthreads();
    int sel_prefix = 0, sel_total = 0;
#pragma unroll
    for (int x = 0; x < NW; ++x) {
      const int v = wsum[NW + x];
      sel_prefix += x < wv ? v : 0;
      sel_total += v;
    }
    if (sel) emit(base_out + sel_prefix + __popcll(bsel & lanemask_lt()), i);
    base_eq += eq_total;
    base_out += sel_total;
    // (no barrier: the next chunk writes wsum[wv] after every wave has passed this chunk's second
    // barrier, so after all reads of wsum[0..NW), and wsum[NW + wv] after its own first barrier)
  }
  return base_out;
}

__device__ int block_count_nonzero(const uint32_t* keys, int n, int* wsum) {
  int c = 0;
  for (int i = threadIdx.x; i < n; i += blockDim.x) c += keys[i] != 0u;
  c = wave_sum(c);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = c;
  __syncthreads();
  int tot = 0;
  for (int x = 0; x < (int)(blockDim.x >> 6); ++x) tot += wsum[x];
  __syncthreads();
  return tot;
}

// Exclusive prefix over NT threads of one value each (sum over threads < t); wtot is LDS [NT/64].
// One block barrier: the caller does not write wtot again before another barrier.
template <int NT, typename V>
__device__ __forceinline__ V block_excl_prefix(V v, V* wtot) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  V inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const V t = __shfl_up(inc, o);
    if (lane >= o) inc += t;
  }
  if (lane == 63) wtot[wv] = inc;
  __syncthreads();
  V base = 0;
#pragma unroll
  for (int x = 0; x < NT / 64; ++x) base += x < wv ? wtot[x] : V(0);
  return base + inc - v;
}

// Reduction over the whole wave without LDS traffic: DPP exchanges within quads (lanes l^1, l^2),
// half rows and rows (mirrors), then gfx950's row swaps (lanes l^16, l^32). op must be commutative
// and associative; every lane ends with the result.
template <typename Op>
__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v, Op op) {
  v = op(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false));   // quad_perm [1, 0, 3, 2]
  v = op(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false));   // quad_perm [2, 3, 0, 1]
  v = op(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x141, 0xF, 0xF, false));  // row_half_mirror
  v = op(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x140, 0xF, 0xF, false));  // row_mirror
  const auto a = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = op(a[0], a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return op(b[0], b[1]);
}
// Number, smallest and largest of the non-zero keys of the block (each(fn) visits this thread's
// keys). One block barrier, which also publishes whatever the caller wrote to LDS before the call;
// wsum, wlo, whi ([NT/64] each) are next written by the caller only after another barrier.
template <int NT, typename Each>
__device__ __forceinline__ void block_nonzero_range(Each&& each, int* wsum, uint32_t* wlo, uint32_t* whi, int& nv,
                                                    uint32_t& lo, uint32_t& hi) {
  uint32_t nz = 0, mn = ~0u, mx = 0u;
  each([&](uint32_t key) {
    if (key != 0u) {
      ++nz;
      mn = key < mn ? key : mn;
      mx = key > mx ? key : mx;
    }
  });
  nz = wave_reduce_u32(nz, [](uint32_t p, uint32_t q) { return p + q; });
  mn = wave_reduce_u32(mn, [](uint32_t p, uint32_t q) { return p < q ? p : q; });
  mx = wave_reduce_u32(mx, [](uint32_t p, uint32_t q) { return p > q ? p : q; });
  if ((threadIdx.x & 63) == 0) {
    wsum[threadIdx.x >> 6] = (int)nz;
    wlo[threadIdx.x >> 6] = mn;
    whi[threadIdx.x >> 6] = mx;
  }
  __syncthreads();
  nv = 0;
  lo = ~0u;
  hi = 0u;
#pragma unroll
  for (int x = 0; x < NT / 64; ++x) {
    nv += wsum[x];
    lo = wlo[x] < lo ? wlo[x] : lo;
    hi = whi[x] > hi ? whi[x] : hi;
  }
}

// Threshold of the k largest non-zero keys of a row held in registers (KPT per thread): T and take
// such that the selection is every key > T and the first `take` keys == T (position order), as
// radix_threshold gives. Each pass counts the keys still in question, those in [lo, hi], into
// kRangeBins bins that split that interval evenly (bin = (key - lo) * scale / 2^32, non-decreasing
// in the key), so one row's scores spread over the bins however closely they cluster, and one
// wave finds the bin holding the rem-th largest key. At most 64 keys in that bin: they are gathered
// into LDS and that wave ranks them against each other. More: the next pass narrows [lo, hi] to the
// smallest and largest key of the bin. A bin spans at most (hi - lo + 1) / 511 + 2 values, so the
// fourth pass sees fewer than kRangeBins values and gives each value its own bin. The scan and the
// ranking are per-row work done once, by wave 0: with several rows per CU the other waves' wait at
// the barrier costs less than eight waves repeating them. lo >= 1 (the smallest non-zero key), so
// key - lo <= hi - lo excludes the zero keys (no candidate) as well as keys outside [lo, hi].
// hist[0 .. 2 kRangeBins) is zero on entry; aux[0] (gathered count) is 0, aux[6], aux[8] (bin
// minimum slots) are ~0u and aux[7], aux[9] (bin maximum slots) 0. Needs rem in [1, keys in play].
constexpr int kRangeBins = 512;
constexpr int kRangeAux = 10;
// each(fn) calls fn(key) for every key this thread holds.
template <int NT, typename Each>
__device__ __forceinline__ void range_threshold(Each&& each, uint32_t lo, uint32_t hi, int rem, uint32_t* hist,
                                                uint32_t* cand, uint32_t* aux, uint32_t& T, int& take) {
  static_assert(kRangeBins == 8 * 64, "a lane scans eight bins");
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  for (int pass = 0; pass < 4; ++pass) {
    uint32_t* hb = hist + kRangeBins * (pass & 1);
    if (pass > 0)  // the other buffer was last read before the previous pass's second barrier
      for (int i = threadIdx.x; i < kRangeBins; i += NT) hist[kRangeBins * ((pass + 1) & 1) + i] = 0u;
    const uint32_t range = hi - lo;
    const bool direct = range < (uint32_t)kRangeBins;  // one value per bin
    // scale <= 512 * 2^32 / (range + 1), so that bins stay below 512 (range >= 512: it fits 32 bits)
    const uint32_t scale = direct ? 0u : (uint32_t)floor(2199023255552.0 / ((double)range + 1.0)) - 1u;
    if (direct)
      each([&](uint32_t key) {
        if (key - lo <= range) atomicAdd(&hb[key - lo], 1u);
      });
    else
      each([&](uint32_t key) {
        if (key - lo <= range) atomicAdd(&hb[__umulhi(key - lo, scale)], 1u);
      });
    __syncthreads();
    if (wv == 0) {
      // lane l holds bins 8 l .. 8 l + 7; keys in the bins of higher lanes by a suffix sum
      const u32x4 ca = reinterpret_cast<const u32x4*>(hb)[2 * lane];
      const u32x4 cb = reinterpret_cast<const u32x4*>(hb)[2 * lane + 1];
      const uint32_t c[8] = {ca.x, ca.y, ca.z, ca.w, cb.x, cb.y, cb.z, cb.w};
      uint32_t tot = 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) tot += c[u];
      uint32_t suf = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t x = __shfl_down(suf, o);
        if (lane + o < 64) suf += x;
      }
      uint32_t above = suf - tot;
#pragma unroll
      for (int u = 7; u >= 0; --u) {
        if (above < (uint32_t)rem && above + c[u] >= (uint32_t)rem) {
          aux[1] = 8 * lane + u;
          aux[2] = above;
          aux[3] = c[u];
        }
        above += c[u];
      }
      if (lane == 0) {  // the other parity's bin extrema were last read before this pass's first barrier
        aux[6 + 2 * ((pass + 1) & 1)] = ~0u;
        aux[7 + 2 * ((pass + 1) & 1)] = 0u;
      }
    }
    __syncthreads();
    const uint32_t bb = aux[1], bc = aux[3];
    rem -= (int)aux[2];
    if (direct) {  // (uniform) the bin is one key value
      T = lo + bb;
      take = rem;
      return;
    }
    auto in_bin = [&](uint32_t key) { return key - lo <= range && __umulhi(key - lo, scale) == bb; };
    if (bc <= 64u) {  // (uniform)
      each([&](uint32_t key) {
        if (in_bin(key)) cand[atomicAdd(&aux[0], 1u)] = key;
      });
      __syncthreads();
      if (wv == 0) {
        // lane l ranks candidate l against all of them: the rem-th largest value has fewer than rem
        // candidates above it and at least rem at or above it; take = rem - (candidates above it)
        const int nb = (int)bc;
        const uint32_t x = cand[lane];  // (lanes >= nb read stale entries and are ignored)
        int gt = 0, ge = 0;
        for (int j = 0; j < nb; j += 4) {
          const u32x4 c4 = *reinterpret_cast<const u32x4*>(cand + j);  // (the same address in every lane)
          const uint32_t cc[4] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const bool in = j + u < nb;
            gt += in && cc[u] > x;
            ge += in && cc[u] >= x;
          }
        }
        const bool hit = lane < nb && gt < rem && ge >= rem;
        if (hit && lane == __ffsll(__ballot(hit)) - 1) {
          aux[4] = x;
          aux[5] = (uint32_t)(rem - gt);
        }
      }
      __syncthreads();
      T = aux[4];
      take = (int)aux[5];
      return;
    }
    // narrow [lo, hi] to the boundary bin's keys
    uint32_t mn = ~0u, mx = 0u;
    each([&](uint32_t key) {
      if (in_bin(key)) {
        mn = key < mn ? key : mn;
        mx = key > mx ? key : mx;
      }
    });
    mn = wave_reduce_u32(mn, [](uint32_t p, uint32_t q) { return p < q ? p : q; });
    mx = wave_reduce_u32(mx, [](uint32_t p, uint32_t q) { return p > q ? p : q; });
    uint32_t* mm = aux + 6 + 2 * (pass & 1);
    if (lane == 0) {
      atomicMin(&mm[0], mn);
      atomicMax(&mm[1], mx);
    }
    __syncthreads();
    lo = mm[0];
    hi = mm[1];
  }
  T = lo;  // (not reached: the fourth pass is direct)
  take = rem;
}

// ============================================================================ Stage 1: page top-M
// Eq. (10): P_t = the M eligible pages of largest coarse score (ties to the smaller page),
// written in ascending page order and padded with -1. All eligible pages when there are <= M.
// Decode (paged cache) also writes, for the k-th recalled page, its physical page (-1 when the
// page-table entry is out of range) to phys[row * ld + k], in the row's own page-key area: the
// fine stage then reads page and physical page side by side instead of a page-table lookup that
// waits for the page. The page-table entries of every eligible page are read into LDS together
// with the page keys, so the lookup adds no round trip here either. (phys aliases page_keys: each
// workgroup reads its row's keys into LDS before its first barrier and writes phys after it.)
template <int NT>
__global__ __launch_bounds__(NT) void page_select_kernel(IndexGeom g, int64_t n_rows, const uint32_t* page_keys,
                                                         int64_t ld, int32_t* __restrict__ pages, int32_t* phys) {
  extern __shared__ uint32_t smem[];
  __shared__ uint32_t hist[2 * kRangeBins];
  __shared__ __align__(16) uint32_t cand[64];
  __shared__ uint32_t aux[kRangeAux];
  __shared__ uint64_t wtot[NT / 64];
  __shared__ int wsum[NT / 64];
  __shared__ uint32_t wlo[NT / 64], whi[NT / 64];
  const int64_t row = blockIdx.x;
  const RowInfo ri = row_info(g, row);
  int32_t* out = pages + row * g.M;
  int32_t* pout = phys ? phys + row * ld : nullptr;
  const int64_t n_elig = (ri.valid && ri.p_hi >= ri.p_lo) ? ri.p_hi - ri.p_lo + 1 : 0;
  if (n_elig <= g.M) {
    for (int i = threadIdx.x; i < g.M; i += NT) out[i] = i < n_elig ? (int32_t)(ri.p_lo + i) : -1;
    if (pout)
      for (int i = threadIdx.x; i < n_elig; i += NT) pout[i] = (int32_t)phys_page(g, row, ri.p_lo + i);
    return;
  }
  const int n = (int)n_elig;
  uint32_t* keys = smem;
  int32_t* ptab = reinterpret_cast<int32_t*>(smem + n);  // decode: physical pages of the eligible pages
  for (int i = threadIdx.x; i < 2 * kRangeBins; i += NT) hist[i] = 0u;
  if (threadIdx.x < kRangeAux) aux[threadIdx.x] = (threadIdx.x == 6 || threadIdx.x == 8) ? ~0u : 0u;
  for (int i = threadIdx.x; i < n; i += NT) {
    keys[i] = page_keys[row * ld + ri.p_lo + i];
    if (pout) ptab[i] = (int32_t)phys_page(g, row, ri.p_lo + i);
  }
  __syncthreads();
  // thread x holds the contiguous slice [x E, x E + E) of the row's page keys
  const int E = (n + NT - 1) / NT;
  const int b = (int)threadIdx.x * E, e = b + E < n ? b + E : n;
  auto each = [&](auto&& fn) {
    for (int i = b; i < e; ++i) fn(keys[i]);
  };
  int nv;
  uint32_t lo, hi;
  block_nonzero_range<NT>(each, wsum, wlo, whi, nv, lo, hi);
  // the M-th largest key: among the non-zero ones, or 0 (pages without a score, taken first to last)
  uint32_t T = 0;
  int take = g.M - nv;
  if (nv > g.M) range_threshold<NT>(each, lo, hi, g.M, hist, cand, aux, T, take);  // (uniform)
  else take = take > 0 ? take : 0;
  // ordered compaction of the slices: (count above T, count equal to T) per thread, one block scan
  uint32_t gt = 0, eq = 0;
  each([&](uint32_t key) {
    gt += key > T;
    eq += key == T;
  });
  const uint64_t pre = block_excl_prefix<NT>((uint64_t)gt | ((uint64_t)eq << 32), wtot);
  const int eq_before = (int)(pre >> 32);
  int rank = (int)(uint32_t)pre + (eq_before < take ? eq_before : take);
  int eqr = eq_before;
  for (int i = b; i < e; ++i) {
    const uint32_t key = keys[i];
    const bool is_eq = key == T;
    if (key > T || (is_eq && eqr < take)) {
      if (pout) pout[rank] = ptab[i];
      out[rank++] = (int32_t)(ri.p_lo + i);
    }
    eqr += is_eq;
  }
}

// ============================================================================ Stage 2: fine token scores
// Eq. (11) over the recalled pages (Eq. 1 over E_t in flat mode), decode variant (paged cache).
// Grid: (n_rows, chunks of pages_per_wg pages); each wave scores whole pages in 32-token MFMA
// tiles. Output: fine_keys[row * ldf + k * P + offset] = order key of the score of position
// page_k * P + offset, or 0 for positions outside E_t.
// Hierarchical mode reads the k-th recalled page from pages[row * M + k] and its physical page
// from phys[row * ldp + k] (written by the page selection); flat mode (phys == nullptr) takes the
// eligible pages in order and looks their physical pages up in the page table. The page ids, the
// physical pages and the query are requested before the row's context length is known (every
// such read stays inside its array), so that the first key tile waits for one round trip after
// them, not for a chain of context length, page, page-table entry and keys.
template <int D, bool FP8>
__global__ __launch_bounds__(256) void fine_kernel(IndexGeom g, int64_t n_rows, const uint16_t* __restrict__ q,
                                                   const float* __restrict__ w, const void* __restrict__ k,
                                                   const float* __restrict__ kscale, const int32_t* __restrict__ pages,
                                                   const int32_t* __restrict__ phys, int64_t ldp,
                                                   uint32_t* __restrict__ fine_keys, int64_t ldf, int pages_per_wg) {
  constexpr int KS = D / 16;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, j = lane & 31;
  const int64_t row = blockIdx.x;
  const bool flat = g.M <= 0;
  const int64_t k0 = (int64_t)blockIdx.y * pages_per_wg;
  // this wave's first two pages (every fourth of the chunk, two at a time; see below): ids and
  // physical pages requested up front (slots below min(M, ldp) are inside the row's arrays)
  int32_t pg_pre[2] = {-1, -1}, ph_pre[2] = {-1, -1};
  if (!flat) {
    const int64_t lim = g.M < ldp ? g.M : ldp;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t kk = k0 + wv + 4 * u;
      if (kk < lim) {
        pg_pre[u] = pages[row * g.M + kk];
        ph_pre[u] = phys[row * ldp + kk];
      }
    }
  }
  u32x4 a[KS];
  float wr[16];
  load_query_operand<D>(q, g.H, row, lane, a);
  load_head_weights(w, g.H, row, lane, wr);

  const RowInfo ri = row_info(g, row);
  if (!ri.valid || ri.p_hi < ri.p_lo) return;
  const int64_t n_elig = ri.p_hi - ri.p_lo + 1;
  const int64_t n_sel = flat ? n_elig : (n_elig < g.M ? n_elig : g.M);
  const int64_t k1 = k0 + pages_per_wg < n_sel ? k0 + pages_per_wg : n_sel;
  if (k0 >= k1) return;

  i32x8 qh[D / 64], ql[D / 64];
  if constexpr (FP8) query_fp8<D>(a, lane, qh, ql, wr);

  constexpr int RAWN = FP8 ? D / 32 : D / 16;  // 16-byte loads per lane per tile
  auto fetch = [&](int64_t kr, u32x4 (&r)[RAWN], float& scl) {
    const u32x4* pp = reinterpret_cast<const u32x4*>(reinterpret_cast<const uint8_t*>(k) + kr * (FP8 ? D : 2 * D) +
                                                    (FP8 ? D / 2 : D) * (lane >> 5));
#pragma unroll
    for (int v = 0; v < RAWN; ++v) r[v] = pp[v];
    scl = FP8 ? kscale[kr] : 1.f;
  };
  const int tpp = g.P / 32;  // 32-token tiles per page
  // the wave's pages (every fourth of the chunk) two at a time: both pages' first key rows are
  // resolved before any key is loaded, then their (page, tile) items are scored in turn with the
  // next item's keys in flight, so the second page's lookups overlap the first page's scoring
  for (int64_t kk0 = k0 + wv; kk0 < k1; kk0 += 8) {
    int64_t pg[2], kb[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t kk = kk0 + 4 * u;
      int64_t ph = -1;
      pg[u] = -1;
      if (kk < k1) {
        if (flat) {
          pg[u] = ri.p_lo + kk;
        } else if (kk0 == k0 + wv) {  // the pair requested up front
          pg[u] = pg_pre[u];
          ph = ph_pre[u];
        } else {
          pg[u] = pages[row * g.M + kk];
          ph = phys[row * ldp + kk];
        }
      }
      kb[u] = -1;  // key row of the page's first token
      if (pg[u] >= ri.p_lo && pg[u] <= ri.p_hi) {
        if (flat) ph = phys_page(g, row, pg[u]);
        kb[u] = ph >= 0 ? ph * g.kv_page : -1;
      }
    }
    const int n_items = (kk0 + 4 < k1 ? 2 : 1) * tpp;
    // key row of lane j in `item` (row 0, not scored, outside E_t or the cache)
    auto krow_of = [&](int item, bool& ok) -> int64_t {
      const int u = item >= tpp, tile = item - u * tpp;
      const int64_t page = u ? pg[1] : pg[0], kbase = u ? kb[1] : kb[0];
      const int64_t pos = page * g.P + tile * 32 + j;
      ok = kbase >= 0 && pos >= ri.lo && pos <= ri.hi;
      return ok ? kbase + tile * 32 + j : 0;
    };
    bool ok;
    u32x4 raw[RAWN];
    float sc;
    fetch(krow_of(0, ok), raw, sc);
    for (int item = 0; item < n_items; ++item) {
      bool nok = false;
      u32x4 nraw[RAWN];
      float nsc = 1.f;
      if (item + 1 < n_items) fetch(krow_of(item + 1, nok), nraw, nsc);  // in flight while this tile is scored
      f32x16 acc = {};
      if constexpr (FP8) {
#pragma unroll
        for (int i = 0; i < D / 64; ++i) {
          const i32x8 b = join_fp8x32(raw[2 * i], raw[2 * i + 1]);
          acc = mfma32_fp8(qh[i], b, acc);
          acc = mfma32_fp8(ql[i], b, acc);
        }
      } else {
#pragma unroll
        for (int s = 0; s < KS; ++s) acc = mfma32(a[s], raw[s], acc);
      }
      float v = head_reduce(acc, wr);
      if (FP8) v *= sc;
      const int u = item >= tpp, tile = item - u * tpp;
      if (lane < 32) fine_keys[row * ldf + (kk0 + 4 * u) * g.P + tile * 32 + j] = ok ? score_key(v) : 0u;
      ok = nok;
      sc = nsc;
#pragma unroll
      for (int e = 0; e < RAWN; ++e) raw[e] = nraw[e];
    }
  }
}

// Prefill variant (contiguous keys): one wave per (group of rows, XCD), the rows taken in turn.
// Workgroup b runs on XCD b mod 8, and the wave of XCD x scores only the recalled pages p with
// p mod 8 == x, so each XCD's L2 holds one eighth of the keys instead of streaming all of them. A page's keys are one contiguous
// block of P rows, copied into LDS 64 rows at a time by direct loads in which the 16-byte granules
// of one key row go to consecutive lanes (a few cache lines per load instead of one line per
// lane); granule c of row t is stored at slot c ^ swz(t) so that the operand reads are
// conflict-free. The two 32-key tiles of a chunk run as two independent MFMA chains.
// Output layout as fine_kernel.
template <int D, bool FP8>
__device__ __forceinline__ int fine_swz(int t) {
  constexpr int RB = FP8 ? D : 2 * D;  // key row bytes
  constexpr int GR = RB / 16;          // 16-byte granules per row
  return RB >= 128 ? (t & 7) : ((t >> (7 - __builtin_ctz(RB))) & (GR - 1));
}

constexpr int kFineChunk = 64;  // key rows staged in LDS at a time
constexpr int kFineRowsPerWave = 8;  // query rows a fine-scoring wave takes in turn

template <int D, bool FP8>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(FP8 || D == 64 ? 4 : 3, 8))) void fine_xcd_kernel(IndexGeom g, int64_t n_rows, const uint16_t* __restrict__ q,
                                                      const float* __restrict__ w, const void* __restrict__ k,
                                                      const float* __restrict__ kscale, const int32_t* __restrict__ pages,
                                                      uint32_t* __restrict__ fine_keys, int64_t ldf) {
  constexpr int KS = D / 16;          // MFMA k-steps
  constexpr int RB = FP8 ? D : 2 * D;
  constexpr int GR = RB / 16;
  constexpr int LG = FP8 ? D / 32 : D / 16;  // 16-byte granules per lane per tile
  __shared__ __attribute__((aligned(16))) uint8_t fsm[kFineChunk * RB];
  __shared__ float lsc[kFineChunk];
  const int lane = threadIdx.x, j = lane & 31, h = lane >> 5;
  const int x = (int)(blockIdx.x & 7);
  // kFineRowsPerWave consecutive query rows, one after the other (fewer, longer-lived waves)
  const int64_t rbeg = (int64_t)(blockIdx.x >> 3) * kFineRowsPerWave;
  const int64_t rend = rbeg + kFineRowsPerWave < n_rows ? rbeg + kFineRowsPerWave : n_rows;
  for (int64_t row = rbeg; row < rend; ++row) {
    const RowInfo ri = row_info(g, row);
    if (!ri.valid || ri.p_hi < ri.p_lo) continue;
    const int64_t n_elig = ri.p_hi - ri.p_lo + 1;
    const bool flat = g.M <= 0;
    const int n_sel = (int)(flat ? n_elig : (n_elig < g.M ? n_elig : g.M));
    const int P = g.P;

    u32x4 a[KS];
    float wr[16];
    load_query_operand<D>(q, g.H, row, lane, a);
    load_head_weights(w, g.H, row, lane, wr);
    i32x8 qh[D / 64], ql[D / 64];
    if constexpr (FP8) query_fp8<D>(a, lane, qh, ql, wr);
    const uint8_t* kb = reinterpret_cast<const uint8_t*>(k);
    uint32_t* const out_row = fine_keys + row * ldf;
    auto tiles_of = [&](int c0) { return P - c0 < kFineChunk ? (P - c0) / 32 : kFineChunk / 32; };  // 1 or 2
    // LDS layout of a chunk: row-major key rows, 16-byte granule c of row t at granule c ^ swz(t)
    // (conflict-free reads of one granule by 8 consecutive rows). Load m fills slots 64 m + lane;
    // src_off(s) is the byte offset, in the chunk's rows, of what slot s holds. It repeats with
    // period 128 slots up to a multiple of 2048 bytes, so two per-lane offsets serve every load.
    auto src_off = [](int s) { const int t = s / GR; return t * RB + 16 * ((s % GR) ^ fine_swz<D, FP8>(t)); };
    const uint32_t voff0 = (uint32_t)src_off(lane), voff1 = (uint32_t)src_off(64 + lane);
    const uint32_t rd0 = (uint32_t)(j * RB + 16 * ((LG * h) ^ fine_swz<D, FP8>(j)));
    const uint32_t lds0 = lds_addr(fsm), lsc0 = lds_addr(lsc);
    // Key rows pg*P + c0 .. + 32 nt - 1 -> the LDS chunk buffer (rows past the last cached key,
    // possible in flat mode when K_swa < P, re-read the last key; their positions get no score).
    auto issue = [&](int64_t pg, int c0) {
      const int nt = tiles_of(c0);
      const int64_t r0 = pg * P + c0;
      if (r0 + 32 * nt <= g.n_kv) {
        const uint8_t* sb = kb + r0 * RB;
  #pragma unroll
        for (int m = 0; m < GR; ++m)
          if (m < GR / 2 || nt == 2) lds_dma<16>(sb + 2048 * (m / 2), (m & 1) ? voff1 : voff0, lds0 + 1024 * m);
        if (FP8 && lane < 32 * nt) lds_dma<4>(kscale + r0, 4u * lane, lsc0);
      } else {
        const int64_t rb = r0 < g.n_kv ? r0 : g.n_kv - 1;  // base row; per-lane rows are clamped to >= it
        const int rmax = (int)(g.n_kv - 1 - rb), rd = (int)(r0 - rb);
        const uint8_t* sb = kb + rb * RB;
        for (int m = 0; m < nt * GR / 2; ++m) {
          const int s = 64 * m + lane, t = s / GR, c = (s % GR) ^ fine_swz<D, FP8>(t);
          const int tr = rd + t < rmax ? rd + t : rmax;
          lds_dma<16>(sb, (uint32_t)(tr * RB + 16 * c), lds0 + 1024 * m);
        }
        const int tr = rd + lane < rmax ? rd + lane : rmax;
        if (FP8 && lane < 32 * nt) lds_dma<4>(kscale + rb, (uint32_t)(4 * tr), lsc0);
      }
    };

    // Pipeline over this wave's work items (page, 64-key chunk): the chunk is read from LDS into
    // registers, the copy of the next chunk into the same buffer starts, and the current one is
    // scored meanwhile. Scores are stored one item late, so that a store has a whole item's compute
    // to complete before the next wait on the memory counter (which counts stores too).
    for (int base = 0; base < n_sel; base += 64) {
      const int kk = base + lane;
      // page ids fit in 31 bits (n_kv < 2^31)
      const int page = kk < n_sel ? (flat ? (int)(ri.p_lo + kk) : pages[row * g.M + kk]) : -1;
      // this wave's pages in this block (recalled pages are always eligible; checked anyway)
      const uint64_t mine = __ballot(page >= ri.p_lo && page <= ri.p_hi && (page & 7) == x);
      if (!mine) continue;
      // page id held by lane b, as a wave-uniform value
      auto page_of = [&](int b) { return (int64_t)__builtin_amdgcn_readlane(page, b); };
      int bit = __builtin_ctzll(mine), c0 = 0;
      issue(page_of(bit), 0);
      uint32_t* pdst = nullptr;                   // pending scores: destination, tiles, values
      int pnt = 0;
      uint32_t pk0 = 0, pk1 = 0;
      while (true) {
        int nbit = bit, nc0 = c0 + kFineChunk;
        bool has_next = true;
        if (nc0 >= P) {
          const uint64_t rest = mine & ~((2ull << bit) - 1ull);  // (2 << 63 wraps to 0: rest = 0)
          has_next = rest != 0;
          nbit = has_next ? __builtin_ctzll(rest) : bit;
          nc0 = 0;
        }
        vm_wait<0>();  // this item's keys (and the previous store) have landed
        const int t0 = j, t1 = 32 + j;
        u32x4 raw0[LG], raw1[LG];
        // granule LG h + v of row j sits at byte rd ^ 16 v (row 32 + j: 32 RB further); rd is
        // re-derived every item so that the compiler keeps one address register, not LG of them
        uint32_t rd = rd0;
        asm volatile("" : "+v"(rd));
  #pragma unroll
        for (int v = 0; v < LG; ++v) {
          raw0[v] = *reinterpret_cast<const u32x4*>(fsm + (rd ^ (16 * v)));
          raw1[v] = *reinterpret_cast<const u32x4*>(fsm + (rd ^ (16 * v)) + 32 * RB);
        }
        const float sc0 = FP8 ? lsc[t0] : 1.f, sc1 = FP8 ? lsc[t1] : 1.f;
        if (pdst != nullptr && lane < 32) {
          pdst[t0] = pk0;
          if (pnt == 2) pdst[t1] = pk1;
        }
        lds_read_wait();  // the buffer may be refilled once every read of it has returned
        if (has_next) issue(page_of(nbit), nc0);
        f32x16 acc0 = {}, acc1 = {};
        if constexpr (FP8) {
  #pragma unroll
          for (int i = 0; i < D / 64; ++i) {
            const i32x8 b0 = join_fp8x32(raw0[2 * i], raw0[2 * i + 1]), b1 = join_fp8x32(raw1[2 * i], raw1[2 * i + 1]);
            acc0 = mfma32_fp8(qh[i], b0, acc0);
            acc1 = mfma32_fp8(qh[i], b1, acc1);
            acc0 = mfma32_fp8(ql[i], b0, acc0);
            acc1 = mfma32_fp8(ql[i], b1, acc1);
          }
        } else {
  #pragma unroll
          for (int s = 0; s < KS; ++s) {
            acc0 = mfma32(a[s], raw0[s], acc0);
            acc1 = mfma32(a[s], raw1[s], acc1);
          }
        }
        // key t of the chunk (position r0 + t) is scored iff lo <= t <= hi (wave-uniform bounds in
        // 32 bits: positions are below n_kv < 2^31)
        const int r0 = (int)page_of(bit) * P + c0;
        const int dlo = (int)ri.lo - r0, dhi = (int)ri.hi - r0;
        const int lo = dlo < 0 ? -1 : (dlo > 64 ? 64 : dlo);
        const int hi = dhi < 0 ? -1 : (dhi > 64 ? 64 : dhi);
        const float v0 = head_reduce(acc0, wr) * sc0;
        const float v1 = head_reduce(acc1, wr) * sc1;
        pk0 = (t0 >= lo && t0 <= hi) ? score_key(v0) : 0u;
        pk1 = (t1 >= lo && t1 <= hi) ? score_key(v1) : 0u;
        pdst = out_row + (int64_t)(base + bit) * P + c0;
        pnt = tiles_of(c0);
        if (!has_next) break;
        bit = nbit;
        c0 = nc0;
      }
      if (lane < 32) {
        pdst[j] = pk0;
        if (pnt == 2) pdst[32 + j] = pk1;
      }
    }
  }
}

// ============================================================================ flat mode: dense causal scoring
// Eq. (7) scored densely (flat mode, prefill). A workgroup of 8 waves takes 8 consecutive query
// rows (wave w: row r0 + w) and walks the block's eligible keys in 64-key chunks, contiguous in the
// cache from the first eligible page on. Each chunk is copied into LDS once (its direct loads spread
// over the 8 waves) and every wave scores it for its own row, so 8 rows share every key byte
// brought on chip. Two LDS buffers: chunk c+1 is copied while chunk c is scored. Output as the fine
// stage's in flat mode: slot s of a row holds position p_lo*P + s, with the order key of its Eq. (1)
// score, or 0 outside the row's eligible range; a row writes its (#eligible pages) * P slots.
constexpr int kFlatRows = 8;  // query rows per workgroup

template <int D, bool FP8>
__global__ __launch_bounds__(64 * kFlatRows) void flat_dense_kernel(IndexGeom g, int64_t n_rows, const uint16_t* __restrict__ q,
                                                                  const float* __restrict__ w, const void* __restrict__ k,
                                                                  const float* __restrict__ kscale,
                                                                  uint32_t* __restrict__ fine_keys, int64_t ldf) {
  constexpr int KS = D / 16;
  constexpr int RB = FP8 ? D : 2 * D;
  constexpr int GR = RB / 16;
  constexpr int LG = FP8 ? D / 32 : D / 16;
  constexpr int CB = kFineChunk * RB;  // bytes of one chunk buffer
  constexpr int NINS = CB / 1024;      // direct loads of 64 x 16 bytes per chunk
  __shared__ __attribute__((aligned(16))) uint8_t fsm[2 * CB];
  __shared__ float lsc[2 * kFineChunk];
  const int lane = threadIdx.x & 63, j = lane & 31, h = lane >> 5;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave index, as a scalar
  const int64_t row0 = (int64_t)blockIdx.x * kFlatRows;
  const int64_t last = row0 + kFlatRows - 1 < n_rows ? row0 + kFlatRows - 1 : n_rows - 1;
  const RowInfo rl = row_info(g, last);  // the block's last row has the longest eligible range
  const int64_t bslots = rl.p_hi >= rl.p_lo ? (rl.p_hi - rl.p_lo + 1) * g.P : 0;
  const int n_chunks = (int)((bslots + kFineChunk - 1) / kFineChunk);
  if (n_chunks == 0) return;  // (uniform over the workgroup)
  const int64_t row = row0 + wv;
  const bool have_row = row < n_rows;
  const RowInfo ri = row_info(g, have_row ? row : last);
  const int64_t nslots = (have_row && ri.p_hi >= ri.p_lo) ? (ri.p_hi - ri.p_lo + 1) * g.P : 0;
  const int64_t base = rl.p_lo * g.P;  // position of slot 0 (p_lo depends on k_sink only)

  u32x4 a[KS];
  float wr[16];
  load_query_operand<D>(q, g.H, have_row ? row : last, lane, a);
  load_head_weights(w, g.H, have_row ? row : last, lane, wr);
  i32x8 qh[D / 64], ql[D / 64];
  if constexpr (FP8) query_fp8<D>(a, lane, qh, ql, wr);
  const uint8_t* kb = reinterpret_cast<const uint8_t*>(k);
  uint32_t* const out_row = fine_keys + (have_row ? row : 0) * ldf;
  // LDS layout of a chunk as in the fine stage (row-major rows, granule c of row t at c ^ swz(t));
  // load m fills slots 64 m + lane, which hold src_off(64 (m % 2) + lane) + 2048 (m / 2) bytes
  // into the chunk's rows
  auto src_off = [](int s) { const int t = s / GR; return t * RB + 16 * ((s % GR) ^ fine_swz<D, FP8>(t)); };
  const uint32_t voff0 = (uint32_t)src_off(lane), voff1 = (uint32_t)src_off(64 + lane);
  const uint32_t rd0 = (uint32_t)(j * RB + 16 * ((LG * h) ^ fine_swz<D, FP8>(j)));
  const uint32_t lds0 = lds_addr(fsm), lsc0 = lds_addr(lsc);
  // chunk c (key positions base + 64 c .. + 63) -> buffer c & 1; this wave's share of the loads.
  // Positions past the cache (a block whose last page is partly cached) re-read the last key.
  auto issue = [&](int c) {
    const int64_t r0 = base + (int64_t)kFineChunk * c;
    const uint32_t lb = lds0 + (uint32_t)((c & 1) * CB);
    if (r0 + kFineChunk <= g.n_kv) {
      const uint8_t* sb = kb + r0 * RB;
      for (int m = wv; m < NINS; m += kFlatRows) lds_dma<16>(sb + 2048 * (m / 2), (m & 1) ? voff1 : voff0, lb + 1024 * m);
      if (FP8 && wv == kFlatRows - 1) lds_dma<4>(kscale + r0, 4u * lane, lsc0 + (uint32_t)((c & 1) * 4 * kFineChunk));
    } else {
      const int64_t rb = r0 < g.n_kv ? r0 : g.n_kv - 1;
      const int rmax = (int)(g.n_kv - 1 - rb), rd = (int)(r0 - rb);
      const uint8_t* sb = kb + rb * RB;
      for (int m = wv; m < NINS; m += kFlatRows) {
        const int sl = 64 * m + lane, t = sl / GR, cc = (sl % GR) ^ fine_swz<D, FP8>(t);
        const int tr = rd + t < rmax ? rd + t : rmax;
        lds_dma<16>(sb, (uint32_t)(tr * RB + 16 * cc), lb + 1024 * m);
      }
      const int tr = rd + lane < rmax ? rd + lane : rmax;
      if (FP8 && wv == kFlatRows - 1)
        lds_dma<4>(kscale + rb, (uint32_t)(4 * tr), lsc0 + (uint32_t)((c & 1) * 4 * kFineChunk));
    }
  };

  issue(0);
  uint32_t pk0 = 0, pk1 = 0;  // scores of the previous chunk, stored one chunk late
  int64_t pslot = -1;
  for (int c = 0; c < n_chunks; ++c) {
    vm_wait_barrier<0>();  // every wave's share of chunk c has landed (and its older stores)
    if (pslot >= 0 && lane < 32) {
      if (pslot + j < nslots) out_row[pslot + j] = pk0;
      if (pslot + 32 + j < nslots) out_row[pslot + 32 + j] = pk1;
    }
    pslot = -1;
    if (c + 1 < n_chunks) issue(c + 1);  // its buffer was last read before this barrier
    const int64_t s0 = (int64_t)kFineChunk * c;
    if (s0 < nslots) {
      const uint8_t* cb = fsm + (c & 1) * CB;
      const float* sb = lsc + (c & 1) * kFineChunk;
      u32x4 raw0[LG], raw1[LG];
      uint32_t rd = rd0;
      asm volatile("" : "+v"(rd));
#pragma unroll
      for (int v = 0; v < LG; ++v) {
        raw0[v] = *reinterpret_cast<const u32x4*>(cb + (rd ^ (16 * v)));
        raw1[v] = *reinterpret_cast<const u32x4*>(cb + (rd ^ (16 * v)) + 32 * RB);
      }
      const float sc0 = FP8 ? sb[j] : 1.f, sc1 = FP8 ? sb[32 + j] : 1.f;
      f32x16 acc0 = {}, acc1 = {};
      if constexpr (FP8) {
#pragma unroll
        for (int i = 0; i < D / 64; ++i) {
          const i32x8 b0 = join_fp8x32(raw0[2 * i], raw0[2 * i + 1]), b1 = join_fp8x32(raw1[2 * i], raw1[2 * i + 1]);
          acc0 = mfma32_fp8(qh[i], b0, acc0);
          acc1 = mfma32_fp8(qh[i], b1, acc1);
          acc0 = mfma32_fp8(ql[i], b0, acc0);
          acc1 = mfma32_fp8(ql[i], b1, acc1);
        }
      } else {
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          acc0 = mfma32(a[s], raw0[s], acc0);
          acc1 = mfma32(a[s], raw1[s], acc1);
        }
      }
      // key t of the chunk (position base + s0 + t) is scored iff lo <= t <= hi
      const int64_t p0 = base + s0;
      const int lo = (int)(ri.lo - p0 < 0 ? -1 : ri.lo - p0 > 64 ? 64 : ri.lo - p0);
      const int hi = (int)(ri.hi - p0 < 0 ? -1 : ri.hi - p0 > 64 ? 64 : ri.hi - p0);
      const float v0 = head_reduce(acc0, wr) * sc0;
      const float v1 = head_reduce(acc1, wr) * sc1;
      pk0 = (j >= lo && j <= hi) ? score_key(v0) : 0u;
      pk1 = (32 + j >= lo && 32 + j <= hi) ? score_key(v1) : 0u;
      pslot = s0;
    }
    lds_read_wait();
  }
  if (pslot >= 0 && lane < 32) {
    if (pslot + j < nslots) out_row[pslot + j] = pk0;
    if (pslot + 32 + j < nslots) out_row[pslot + 32 + j] = pk1;
  }
}

// ============================================================================ final top-K_sparse, merge, runs
// Writes idx/count of one row from lidx[0..cnt) and, if requested, its runs: maximal stretches of
// consecutive positions, also cut at multiples of C. rstart is LDS scratch of >= cnt entries.
template <int NT>
__device__ void emit_row(const IndexGeom& g, int64_t row, const int32_t* lidx, int cnt, int32_t* rstart, int* wsum,
                         int32_t* __restrict__ idx, int32_t* __restrict__ count, int32_t* __restrict__ runs,
                         int32_t* __restrict__ run_count) {
  const int k_cap = g.k_sink + g.k_swa + g.k_sparse;
  int32_t* orow = idx + row * k_cap;
  for (int i = threadIdx.x; i < k_cap; i += NT) orow[i] = i < cnt ? lidx[i] : -1;
  if (threadIdx.x == 0) count[row] = cnt;
  if (!runs) return;
  // A run starts at i = 0, after a gap, or at a position divisible by C. Thread x scans the
  // contiguous slice [x E, x E + E) of the list; one block-wide prefix of the per-thread start
  // counts numbers the runs, and each run is stored as one 8-byte (start, length) pair.
  const int C = g.C;
  const bool c2 = (C & (C - 1)) == 0;  // (uniform) multiples of C by a mask
  auto starts = [&](int i, int32_t s) {
    return i == 0 || s != lidx[i - 1] + 1 || (c2 ? (s & (C - 1)) == 0 : (s % C) == 0);
  };
  const int E = (cnt + NT - 1) / NT;
  const int b = (int)threadIdx.x * E, e = b + E < cnt ? b + E : cnt;
  int mine = 0;
  uint64_t fl = 0;  // start flags of the slice's first 64 entries
  for (int i = b; i < e; ++i)
    if (starts(i, lidx[i])) {
      ++mine;
      fl |= i - b < 64 ? 1ull << (i - b) : 0ull;
    }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int inc = mine;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(inc, o);
    if (lane >= o) inc += t;
  }
  if (lane == 63) wsum[wv] = inc;
  __syncthreads();
  int r = inc - mine, nr = 0;
#pragma unroll
  for (int x = 0; x < NT / 64; ++x) {
    const int v = wsum[x];
    r += x < wv ? v : 0;
    nr += v;
  }
  if (E <= 64) {  // (uniform)
    for (; fl != 0; fl &= fl - 1) rstart[r++] = b + __ffsll((unsigned long long)fl) - 1;
  } else {
    for (int i = b; i < e; ++i)
      if (starts(i, lidx[i])) rstart[r++] = i;
  }
  __syncthreads();
  int2* rrow = reinterpret_cast<int2*>(runs + row * (int64_t)k_cap * 2);  // 8-byte aligned (checked on the host)
  for (int q = threadIdx.x; q < nr; q += NT) {  // entries past run_count are not written
    const int s0 = rstart[q];
    const int s1 = q + 1 < nr ? rstart[q + 1] : cnt;
    rrow[q] = make_int2(lidx[s0], s1 - s0);
  }
  if (threadIdx.x == 0) run_count[row] = nr;
}

// Threshold of the k largest of the n keys of a row held in global memory (see radix_threshold),
// in two passes over them instead of five: an 11-bit histogram of the non-zero keys (counting
// them), then the keys of the bin holding the k-th largest are gathered into LDS, where radix
// passes over the remaining bits finish. When that bin holds more than cap keys, the radix
// passes run over the whole row instead. Returns the non-zero count; T = 0, take_eq = 0 when at
// most k keys are non-zero (every one is selected).
constexpr int kSelHistBits = 11;
constexpr int kSelGatherCap = 8192;

// One streaming pass over a row's n keys in global memory (n a multiple of 32, the row 16-byte
// aligned): wave w takes the contiguous span [w S, w S + S) (S: the row over the NT / 64 waves, in
// stretches of 256 keys), lane l reading keys 4l .. 4l + 3 of each stretch with one 16-byte load,
// four stretches in flight. fn(i, keys i .. i + 3, valid) is called per lane for every stretch of
// the span in increasing order, so a wave visits its span in position order (stretch by stretch,
// lane by lane).
template <int NT, typename F>
__device__ __forceinline__ void stream_row(const uint32_t* keys, int n, F&& fn) {
  constexpr int NW = NT / 64;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int span = (n + NW * 256 - 1) / (NW * 256) * 256;
  const int s0 = wv * span, s1 = s0 + span < n ? s0 + span : n;
  for (int b = s0; b < s1; b += 1024) {
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = b + 256 * u + 4 * lane;
      v[u] = i < s1 ? *reinterpret_cast<const u32x4*>(keys + i) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = b + 256 * u + 4 * lane;
      if (b + 256 * u < s1) fn(i, v[u], i < s1);  // (uniform per wave: the stretch starts in the span)
    }
  }
}

template <int NT>
__device__ int global_threshold(const uint32_t* keys, int n, int k, uint32_t* h11, uint32_t* sub, int* gcnt,
                                uint32_t* hist, int* wsum, uint32_t& T, int& take_eq) {
  constexpr int NB = 1 << kSelHistBits;
  for (int i = threadIdx.x; i < NB; i += NT) h11[i] = 0;
  for (int i = threadIdx.x; i < 256; i += NT) hist[i] = 0;  // (for radix_threshold)
  if (threadIdx.x == 0) *gcnt = 0;
  __syncthreads();
  int nz = 0;
  stream_row<NT>(keys, n, [&](int, const u32x4& v, bool ok) {
    const uint32_t k4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (ok && k4[c] != 0u) {
        atomicAdd(&h11[k4[c] >> (32 - kSelHistBits)], 1u);
        ++nz;
      }
  });
  nz = wave_sum(nz);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = nz;
  __syncthreads();
  int n_valid = 0;
  for (int x = 0; x < NT / 64; ++x) n_valid += wsum[x];
  T = 0;
  take_eq = 0;
  __syncthreads();  // wsum is reused below, and by the caller's compaction
  if (n_valid <= k) return n_valid;  // (uniform)
  // bin b* holding the k-th largest key, and the count of keys in the bins above it
  if (threadIdx.x < 64) {
    constexpr int PER = NB / 64;
    const int l = threadIdx.x;
    uint32_t tot = 0;
    for (int b = 0; b < PER; ++b) tot += h11[PER * l + b];
    uint32_t suf = tot;  // totals of lanes >= l
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t x = __shfl_down(suf, o);
      if (l + o < 64) suf += x;
    }
    uint32_t above = suf - tot;
    if (above < (uint32_t)k && suf >= (uint32_t)k) {
      for (int b = PER - 1; b >= 0; --b) {
        const uint32_t c = h11[PER * l + b];
        if (above + c >= (uint32_t)k) {
          wsum[0] = PER * l + b;
          wsum[1] = (int)above;
          break;
        }
        above += c;
      }
    }
  }
  __syncthreads();
  const uint32_t bstar = (uint32_t)wsum[0];
  const int rem = k - wsum[1];
  // the boundary bin's keys -> LDS (order is irrelevant: only the threshold and the number of
  // ties to take are derived from them; select_compact then takes ties in position order)
  stream_row<NT>(keys, n, [&](int, const u32x4& v, bool ok) {
    const uint32_t k4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (ok && k4[c] != 0u && (k4[c] >> (32 - kSelHistBits)) == bstar) {
        const int at = atomicAdd(gcnt, 1);
        if (at < kSelGatherCap) sub[at] = k4[c];
      }
  });
  __syncthreads();
  const int nb = *gcnt;
  __syncthreads();
  if (nb <= kSelGatherCap) radix_threshold<NT>(sub, nb, rem, hist, T, take_eq, 1);
  else radix_threshold<NT>(keys, n, k, hist, T, take_eq);
  return n_valid;
}

// select_compact for keys in global memory, in two streaming passes: each wave counts its span's
// keys above T and its ties, one block scan of the per-wave counts gives each wave its first output
// rank and the number of ties before its span, and each wave then writes its selected positions in
// position order (wave-wide prefix sums per stretch, no block barrier). Same selection and ranks
// as select_compact; returns the number selected.
template <int NT, typename F>
__device__ int global_compact(const uint32_t* keys, int n, uint32_t T, int take_eq, int* wsum, F&& emit) {
  constexpr int NW = NT / 64;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int gt = 0, eq = 0;
  stream_row<NT>(keys, n, [&](int, const u32x4& v, bool ok) {
    const uint32_t k4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      gt += ok && k4[c] > T;
      eq += ok && k4[c] == T;
    }
  });
  gt = wave_sum(gt);
  eq = wave_sum(eq);
  if (lane == 0) {
    wsum[wv] = gt;
    wsum[NW + wv] = eq;
  }
  __syncthreads();
  int sel_before = 0, eq_before = 0, total = 0, eqb = 0;
#pragma unroll
  for (int x = 0; x < NW; ++x) {
    const int g_ = wsum[x], e_ = wsum[NW + x];
    int t_ = take_eq - eqb;
    t_ = t_ < 0 ? 0 : (t_ > e_ ? e_ : t_);
    if (x < wv) {
      sel_before += g_ + t_;
      eq_before += e_;
    }
    total += g_ + t_;
    eqb += e_;
  }
  __syncthreads();  // (wsum is reused by the caller)
  auto excl = [&](int v, int& tot) {  // exclusive prefix over the lanes, and the wave total
    int inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int t = __shfl_up(inc, o);
      if (lane >= o) inc += t;
    }
    tot = __shfl(inc, 63);
    return inc - v;
  };
  int out = sel_before, eqr = eq_before;
  stream_row<NT>(keys, n, [&](int i, const u32x4& v, bool ok) {
    const uint32_t k4[4] = {v.x, v.y, v.z, v.w};
    int e_l = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) e_l += ok && k4[c] == T;
    int e_tot;
    int er = eqr + excl(e_l, e_tot);
    bool sel[4];
    int s_l = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const bool is_eq = ok && k4[c] == T;
      sel[c] = ok && (k4[c] > T || (is_eq && er < take_eq));
      er += is_eq;
      s_l += sel[c];
    }
    int s_tot;
    int r = out + excl(s_l, s_tot);
#pragma unroll
    for (int c = 0; c < 4; ++c)
      if (sel[c]) emit(r++, i + c);
    out += s_tot;
    eqr += e_tot;
  });
  return total;
}

// Eq. (12) / Eq. (7) then Eq. (6): S_t = sink ++ (top K_sparse candidates, ascending) ++ window;
// idx padded with -1; runs re-encode idx, cut at gaps and at multiples of C. General version:
// the candidate keys are staged in LDS (any number that fits), or with GK (rows too long for
// LDS) every pass reads them from the fine-score rows in global memory.
template <int NT, bool GK>
__global__ __launch_bounds__(NT) void token_select_kernel(IndexGeom g, int64_t n_rows, const uint32_t* __restrict__ fine_keys,
                                                          int64_t ldf, const int32_t* __restrict__ pages,
                                                          int32_t* __restrict__ idx, int32_t* __restrict__ count,
                                                          int32_t* __restrict__ runs, int32_t* __restrict__ run_count,
                                                          int slots_cap) {
  extern __shared__ uint32_t smem[];
  __shared__ uint32_t hist[256];
  __shared__ int wsum[2 * NT / 64 + 2];
  const int k_cap = g.k_sink + g.k_swa + g.k_sparse;
  // LDS: keys [max(slots_cap, k_cap)] (not with GK), lidx [k_cap], lpages [M], and with GK the
  // run-start scratch [k_cap] (otherwise the keys area serves for it), the 11-bit histogram, the
  // gathered boundary-bin keys and their counter
  const int key_words = GK ? 0 : (slots_cap > k_cap ? slots_cap : k_cap);
  int32_t* lidx = reinterpret_cast<int32_t*>(smem + key_words);
  int32_t* lpages = lidx + k_cap;
  int32_t* rstart = GK ? lpages + (g.M > 0 ? g.M : 0) : reinterpret_cast<int32_t*>(smem);
  uint32_t* h11 = reinterpret_cast<uint32_t*>(rstart + k_cap);
  uint32_t* gsub = h11 + (1 << kSelHistBits);
  int* gcnt = reinterpret_cast<int*>(gsub + kSelGatherCap);

  const int64_t row = blockIdx.x;
  const RowInfo ri = row_info(g, row);
  int cnt = 0;
  if (!ri.valid) {
    cnt = 0;
  } else if (ri.p_hi < ri.p_lo) {
    // sink and window cover [0, t]
    cnt = (int)(ri.t + 1);
    for (int i = threadIdx.x; i < cnt; i += NT) lidx[i] = i;
  } else {
    const bool flat = g.M <= 0;
    const int64_t n_elig = ri.p_hi - ri.p_lo + 1;
    const int n_sel = (int)(flat ? n_elig : (n_elig < g.M ? n_elig : g.M));
    if (!flat)
      for (int i = threadIdx.x; i < n_sel; i += NT) lpages[i] = pages[row * g.M + i];
    const int n = n_sel * g.P;
    const uint32_t* keys = GK ? fine_keys + row * ldf : smem;
    if (!GK) {
      for (int i = threadIdx.x; i < 256; i += NT) hist[i] = 0;  // (for radix_threshold)
      for (int i = threadIdx.x; i < n; i += NT) smem[i] = fine_keys[row * ldf + i];
    }
    __syncthreads();
    uint32_t T = 0;
    int take = 0;
    if (GK) {
      global_threshold<NT>(keys, n, g.k_sparse, h11, gsub, gcnt, hist, wsum, T, take);
    } else {
      const int n_valid = block_count_nonzero(keys, n, wsum);
      if (n_valid > g.k_sparse) radix_threshold<NT>(keys, n, g.k_sparse, hist, T, take);
    }
    const int P = g.P;
    const bool p2 = (P & (P - 1)) == 0;  // (uniform) slot -> page by a shift
    const int lgP = __ffs(P) - 1;
    const int64_t p_lo = ri.p_lo;
    const int ks = g.k_sink;
    auto emit = [&](int rank, int i) {
      const int pi = p2 ? i >> lgP : i / P;
      const int64_t page = flat ? p_lo + pi : (int64_t)lpages[pi];
      lidx[ks + rank] = (int32_t)(page * P + (i - pi * P));
    };
    int n_sp;
    if constexpr (GK) n_sp = global_compact<NT>(keys, n, T, take, wsum, emit);
    else n_sp = select_compact<NT>(keys, n, T, take, wsum, emit);
    for (int i = threadIdx.x; i < g.k_sink; i += NT) lidx[i] = i;
    for (int i = threadIdx.x; i < g.k_swa; i += NT) lidx[g.k_sink + n_sp + i] = (int32_t)(ri.t - g.k_swa + 1 + i);
    cnt = g.k_sink + n_sp + g.k_swa;
  }
  __syncthreads();
  emit_row<NT>(g, row, lidx, cnt, rstart, wsum, idx, count, runs, run_count);
}

// Rows of at most 16 keys per thread run eight waves per SIMD (four rows of 512 threads per CU):
// the registers are capped so that the small LDS footprint is what bounds the rows a CU holds.
template <int NT, int KPT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(KPT <= 16 ? 8 : 1))) void token_select_reg_kernel(
    IndexGeom g, int64_t n_rows, const uint32_t* __restrict__ fine_keys, int64_t ldf, const int32_t* __restrict__ pages,
    int32_t* __restrict__ idx, int32_t* __restrict__ count, int32_t* __restrict__ runs, int32_t* __restrict__ run_count) {
  extern __shared__ int32_t dyn[];  // lidx [k_cap], rstart [k_cap], lpages [M]
  __shared__ uint32_t hist[2 * kRangeBins];
  __shared__ __align__(16) uint32_t cand[64];
  __shared__ uint32_t aux[kRangeAux];
  __shared__ uint32_t wtot[NT / 64 + 2];
  __shared__ int wsum[NT / 64 + 2];
  __shared__ uint32_t wlo[NT / 64], whi[NT / 64];
  const int k_cap = g.k_sink + g.k_swa + g.k_sparse;
  int32_t* lidx = dyn;
  int32_t* rstart = dyn + k_cap;
  int32_t* lpages = dyn + 2 * k_cap;

  const int64_t row = blockIdx.x;
  const RowInfo ri = row_info(g, row);
  int cnt = 0;
  if (!ri.valid) {
    cnt = 0;
  } else if (ri.p_hi < ri.p_lo) {
    cnt = (int)(ri.t + 1);  // sink and window cover [0, t]
    for (int i = threadIdx.x; i < cnt; i += NT) lidx[i] = i;
  } else {
    const bool flat = g.M <= 0;
    const int64_t n_elig = ri.p_hi - ri.p_lo + 1;
    const int n_sel = (int)(flat ? n_elig : (n_elig < g.M ? n_elig : g.M));
    if (!flat)
      for (int i = threadIdx.x; i < n_sel; i += NT) lpages[i] = pages[row * g.M + i];
    const int n = n_sel * g.P;
    for (int i = threadIdx.x; i < 2 * kRangeBins; i += NT) hist[i] = 0u;
    if (threadIdx.x < kRangeAux) aux[threadIdx.x] = (threadIdx.x == 6 || threadIdx.x == 8) ? ~0u : 0u;
    const int i0 = (int)threadIdx.x * KPT;
    uint32_t kv[KPT];
    const uint32_t* src = fine_keys + row * ldf + i0;
#pragma unroll
    for (int e = 0; e < KPT; e += 4) {
      if (i0 + e + 4 <= n) {
        const u32x4 v = *reinterpret_cast<const u32x4*>(src + e);
        kv[e] = v.x; kv[e + 1] = v.y; kv[e + 2] = v.z; kv[e + 3] = v.w;
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) kv[e + u] = i0 + e + u < n ? src[e + u] : 0u;
      }
    }
    auto each = [&](auto&& fn) {
#pragma unroll
      for (int e = 0; e < KPT; ++e) fn(kv[e]);
    };
    // non-zero keys (the candidates), their smallest and their largest; the barrier also publishes
    // the cleared histograms and aux
    int nv;
    uint32_t lo, hi;
    block_nonzero_range<NT>(each, wsum, wlo, whi, nv, lo, hi);
    uint32_t T = 0;
    int take = 0;
    if (nv > g.k_sparse) range_threshold<NT>(each, lo, hi, g.k_sparse, hist, cand, aux, T, take);  // (uniform)
    // ordered compaction: selected = key > T, or key == T among the first `take` such (index order);
    // with T = 0 (every candidate selected) take is 0, so counting the zero keys as ties is harmless
    uint32_t gt = 0, eq = 0;
#pragma unroll
    for (int e = 0; e < KPT; ++e) {
      gt += kv[e] > T;
      eq += kv[e] == T;
    }
    const uint32_t pre = block_excl_prefix<NT>(gt | (eq << 16), wtot);
    const int eq_before = (int)(pre >> 16);
    int out = (int)(pre & 0xFFFFu) + (eq_before < take ? eq_before : take);
    int eqr = eq_before;
    const int P = g.P, ks = g.k_sink;
    auto pos_of = [&](int i) {
      const int pi = i / P;
      const int64_t page = flat ? ri.p_lo + pi : (int64_t)lpages[pi];
      return (int32_t)(page * P + (i - pi * P));
    };
    if (gt + eq > 0) {  // (P is a multiple of 32: a thread's KPT <= 32 keys lie in one page)
      const int32_t base = KPT <= 32 || P % KPT == 0 ? pos_of(i0) : 0;
#pragma unroll
      for (int e = 0; e < KPT; ++e) {
        const uint32_t key = kv[e];
        const bool is_eq = key == T;
        const bool sel = key > T || (is_eq && eqr < take);
        eqr += is_eq;
        if (sel) lidx[ks + out++] = KPT <= 32 || P % KPT == 0 ? base + e : pos_of(i0 + e);
      }
    }
    const int n_sp = nv > g.k_sparse ? g.k_sparse : nv;
    for (int i = threadIdx.x; i < g.k_sink; i += NT) lidx[i] = i;
    for (int i = threadIdx.x; i < g.k_swa; i += NT) lidx[g.k_sink + n_sp + i] = (int32_t)(ri.t - g.k_swa + 1 + i);
    cnt = g.k_sink + n_sp + g.k_swa;
  }
  __syncthreads();
  emit_row<NT>(g, row, lidx, cnt, rstart, wsum, idx, count, runs, run_count);
}

// ============================================================================ host launchers
template <bool FP8, bool MINMAX>
static hipError_t launch_bk(int64_t n_items, const int64_t* rows, int64_t n_tok, int D, int B, const void* k,
                            const float* ks, uint16_t* out, hipStream_t st) {
  const int64_t threads = n_items * (D / 4);
  if (threads == 0) return hipSuccess;
  const int64_t blocks = (threads + 255) / 256;
  if (MINMAX)
    hipLaunchKernelGGL(block_minmax_kernel<FP8>, dim3((unsigned)blocks), dim3(256), 0, st, n_items, rows, n_tok, D, B,
                       k, ks, out);
  else
    hipLaunchKernelGGL(block_means_kernel<FP8>, dim3((unsigned)blocks), dim3(256), 0, st, n_items, rows, n_tok, D, B,
                       k, ks, out);
  return hipGetLastError();
}

hipError_t launch_block_keys(int64_t n_items, const int64_t* rows, int64_t n_tok, int D, int B, bool fp8, bool minmax,
                             const void* k, const float* ks, uint16_t* out, hipStream_t st) {
  if (minmax)
    return fp8 ? launch_bk<true, true>(n_items, rows, n_tok, D, B, k, ks, out, st)
               : launch_bk<false, true>(n_items, rows, n_tok, D, B, k, ks, out, st);
  return fp8 ? launch_bk<true, false>(n_items, rows, n_tok, D, B, k, ks, out, st)
             : launch_bk<false, false>(n_items, rows, n_tok, D, B, k, ks, out, st);
}

template <int D, int R, bool PAGED, bool MINMAX>
static hipError_t launch_coarse_t(const IndexGeom& g, int64_t n_rows, const uint16_t* q, const float* w,
                                  const uint16_t* kmean, uint32_t* page_keys, int64_t ld, int64_t max_tiles,
                                  hipStream_t st) {
  if (max_tiles <= 0 || n_rows == 0) return hipSuccess;
  if (!PAGED && !MINMAX && max_tiles <= kCoarseStagedTiles && g.n_sub > 0 &&
      g.n_sub <= ((int64_t)1 << 32) / D / 2) {  // one wave per workgroup, all tiles of its rows
    constexpr int RS = kCoarseRowsStaged;
    const dim3 grid((unsigned)((n_rows + RS - 1) / RS), 1u);
    hipLaunchKernelGGL((coarse_kernel<D, RS, false, false, true>), grid, dim3(64), 0, st, g, n_rows, q, w, kmean,
                       page_keys, ld, (int)max_tiles);
    return hipGetLastError();
  }
  const int tiles_per_chunk = PAGED ? 8 : (int)max_tiles;
  const int64_t chunks = (max_tiles + tiles_per_chunk - 1) / tiles_per_chunk;
  const dim3 grid((unsigned)((n_rows + R - 1) / R), (unsigned)chunks);
  hipLaunchKernelGGL((coarse_kernel<D, R, PAGED, MINMAX>), grid, dim3(256), 0, st, g, n_rows, q, w, kmean, page_keys,
                     ld, tiles_per_chunk);
  return hipGetLastError();
}

template <int D, bool MINMAX>
static hipError_t launch_coarse_d(const IndexGeom& g, int64_t n_rows, const uint16_t* q, const float* w,
                                  const uint16_t* kmean, uint32_t* page_keys, int64_t ld, int64_t max_tiles,
                                  hipStream_t st) {
  // min-max doubles the operands' width: fewer query rows share a tile (register budget)
  constexpr int R = MINMAX ? 2 : 4;
  return g.ctx_len != nullptr ? launch_coarse_t<D, 1, true, MINMAX>(g, n_rows, q, w, kmean, page_keys, ld, max_tiles, st)
                              : launch_coarse_t<D, R, false, MINMAX>(g, n_rows, q, w, kmean, page_keys, ld, max_tiles, st);
}

hipError_t launch_coarse(const IndexGeom& g, int64_t n_rows, const uint16_t* q, const float* w, const uint16_t* kmean,
                         uint32_t* page_keys, int64_t ld, int64_t max_tiles, hipStream_t st) {
  if (g.D == 128)
    return g.minmax ? launch_coarse_d<128, true>(g, n_rows, q, w, kmean, page_keys, ld, max_tiles, st)
                    : launch_coarse_d<128, false>(g, n_rows, q, w, kmean, page_keys, ld, max_tiles, st);
  return g.minmax ? launch_coarse_d<64, true>(g, n_rows, q, w, kmean, page_keys, ld, max_tiles, st)
                  : launch_coarse_d<64, false>(g, n_rows, q, w, kmean, page_keys, ld, max_tiles, st);
}

hipError_t launch_page_select(const IndexGeom& g, int64_t n_rows, const uint32_t* page_keys, int64_t ld,
                              int32_t* pages, int32_t* phys, int64_t max_elig, hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  const size_t lds = page_select_lds_bytes(max_elig, phys != nullptr);
  if (n_rows <= kSelectFewRows)  // few rows (decode): more threads per row
    hipLaunchKernelGGL(page_select_kernel<1024>, dim3((unsigned)n_rows), dim3(1024), lds, st, g, n_rows, page_keys, ld,
                       pages, phys);
  else
    hipLaunchKernelGGL(page_select_kernel<256>, dim3((unsigned)n_rows), dim3(256), lds, st, g, n_rows, page_keys, ld,
                       pages, phys);
  return hipGetLastError();
}

template <int D, bool FP8>
static hipError_t launch_fine_t(const IndexGeom& g, int64_t n_rows, const uint16_t* q, const float* w, const void* k,
                                const float* ks, const int32_t* pages, const int32_t* phys, int64_t ldp,
                                uint32_t* fine_keys, int64_t ldf, int64_t max_sel, hipStream_t st) {
  constexpr int ppw = 8;  // recalled pages per workgroup (two per wave)
  const int64_t chunks = (max_sel + ppw - 1) / ppw;
  if (chunks == 0 || n_rows == 0) return hipSuccess;
  hipLaunchKernelGGL((fine_kernel<D, FP8>), dim3((unsigned)n_rows, (unsigned)chunks), dim3(256), 0, st, g, n_rows, q, w,
                     k, ks, pages, phys, ldp, fine_keys, ldf, ppw);
  return hipGetLastError();
}

template <int D, bool FP8>
static hipError_t launch_fine_xcd_t(const IndexGeom& g, int64_t n_rows, const uint16_t* q, const float* w,
                                    const void* k, const float* ks, const int32_t* pages, uint32_t* fine_keys,
                                    int64_t ldf, hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  const int64_t waves_per_xcd = (n_rows + kFineRowsPerWave - 1) / kFineRowsPerWave;
  hipLaunchKernelGGL((fine_xcd_kernel<D, FP8>), dim3((unsigned)(waves_per_xcd * 8)), dim3(64), 0, st, g, n_rows, q, w, k, ks,
                     pages, fine_keys, ldf);
  return hipGetLastError();
}

template <int D, bool FP8>
static hipError_t launch_flat_dense_t(const IndexGeom& g, int64_t n_rows, const uint16_t* q, const float* w,
                                      const void* k, const float* ks, uint32_t* fine_keys, int64_t ldf, hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  hipLaunchKernelGGL((flat_dense_kernel<D, FP8>), dim3((unsigned)((n_rows + kFlatRows - 1) / kFlatRows)),
                     dim3(64 * kFlatRows), 0, st, g, n_rows, q, w, k, ks, fine_keys, ldf);
  return hipGetLastError();
}

hipError_t launch_fine(const IndexGeom& g, int64_t n_rows, const uint16_t* q, const float* w, const void* k,
                       const float* ks, const int32_t* pages, const int32_t* phys, int64_t ldp, uint32_t* fine_keys,
                       int64_t ldf, int64_t max_sel, hipStream_t st) {
  const bool paged = g.ctx_len != nullptr, fp8 = g.fp8 != 0;
  if (!paged && g.M <= 0) {  // flat prefill: dense causal scoring
    if (max_sel <= 0) return hipSuccess;
    if (g.D == 128) return fp8 ? launch_flat_dense_t<128, true>(g, n_rows, q, w, k, ks, fine_keys, ldf, st)
                               : launch_flat_dense_t<128, false>(g, n_rows, q, w, k, ks, fine_keys, ldf, st);
    return fp8 ? launch_flat_dense_t<64, true>(g, n_rows, q, w, k, ks, fine_keys, ldf, st)
               : launch_flat_dense_t<64, false>(g, n_rows, q, w, k, ks, fine_keys, ldf, st);
  }
  if (!paged) {
    if (max_sel <= 0) return hipSuccess;
    if (g.D == 128) return fp8 ? launch_fine_xcd_t<128, true>(g, n_rows, q, w, k, ks, pages, fine_keys, ldf, st)
                               : launch_fine_xcd_t<128, false>(g, n_rows, q, w, k, ks, pages, fine_keys, ldf, st);
    return fp8 ? launch_fine_xcd_t<64, true>(g, n_rows, q, w, k, ks, pages, fine_keys, ldf, st)
               : launch_fine_xcd_t<64, false>(g, n_rows, q, w, k, ks, pages, fine_keys, ldf, st);
  }
  // paged decode: per (sequence, page) through the page table
  if (g.D == 128)
    return fp8 ? launch_fine_t<128, true>(g, n_rows, q, w, k, ks, pages, phys, ldp, fine_keys, ldf, max_sel, st)
               : launch_fine_t<128, false>(g, n_rows, q, w, k, ks, pages, phys, ldp, fine_keys, ldf, max_sel, st);
  return fp8 ? launch_fine_t<64, true>(g, n_rows, q, w, k, ks, pages, phys, ldp, fine_keys, ldf, max_sel, st)
             : launch_fine_t<64, false>(g, n_rows, q, w, k, ks, pages, phys, ldp, fine_keys, ldf, max_sel, st);
}

// Which selection kernel serves rows of slots_cap candidates: keys in registers, staged in LDS,
// or read from global memory in every pass (rows too long for LDS).
enum class SelectMode { kRegisters, kLds, kGlobal };
constexpr size_t kSelectLdsLimit = 160 * 1024 - 4096;  // dynamic LDS the select kernels may use

static SelectMode select_mode(int64_t slots_cap, int k_cap, int M) {
  if (slots_cap <= kSelectRegMax) return SelectMode::kRegisters;
  const int64_t a = slots_cap > k_cap ? slots_cap : k_cap;
  return (size_t)(a + k_cap + (M > 0 ? M : 0)) * 4 <= kSelectLdsLimit ? SelectMode::kLds : SelectMode::kGlobal;
}

size_t token_select_lds_bytes(int64_t slots_cap, int k_cap, int M) {
  const size_t m = (size_t)(M > 0 ? M : 0);
  switch (select_mode(slots_cap, k_cap, M)) {
    case SelectMode::kRegisters: return (2 * (size_t)k_cap + m) * 4;
    case SelectMode::kLds: return ((size_t)(slots_cap > k_cap ? slots_cap : k_cap) + k_cap + m) * 4;
    default: return (2 * (size_t)k_cap + m + (1u << kSelHistBits) + kSelGatherCap + 1) * 4;
  }
}

hipError_t launch_token_select(const IndexGeom& g, int64_t n_rows, const uint32_t* fine_keys, int64_t ldf,
                               const int32_t* pages, int32_t* idx, int32_t* count, int32_t* runs, int32_t* run_count,
                               int64_t slots_cap, hipStream_t st) {
  if (n_rows == 0) return hipSuccess;
  const int k_cap = g.k_sink + g.k_swa + g.k_sparse;
  const size_t lds = token_select_lds_bytes(slots_cap, k_cap, g.M);
  const dim3 grid((unsigned)n_rows), block(512);
  if (slots_cap <= 1024 * 8 && n_rows <= kSelectFewRows)   // few rows (decode): more threads per row
    hipLaunchKernelGGL((token_select_reg_kernel<1024, 8>), grid, dim3(1024), lds, st, g, n_rows, fine_keys, ldf, pages,
                       idx, count, runs, run_count);
  else if (slots_cap <= 512 * 16)
    hipLaunchKernelGGL((token_select_reg_kernel<512, 16>), grid, block, lds, st, g, n_rows, fine_keys, ldf, pages, idx,
                       count, runs, run_count);
  else if (slots_cap <= 512 * 32)
    hipLaunchKernelGGL((token_select_reg_kernel<512, 32>), grid, block, lds, st, g, n_rows, fine_keys, ldf, pages, idx,
                       count, runs, run_count);
  else if (slots_cap <= kSelectRegMax)
    hipLaunchKernelGGL((token_select_reg_kernel<512, 64>), grid, block, lds, st, g, n_rows, fine_keys, ldf, pages, idx,
                       count, runs, run_count);
  else if (select_mode(slots_cap, k_cap, g.M) == SelectMode::kLds)
    hipLaunchKernelGGL((token_select_kernel<512, false>), grid, block, lds, st, g, n_rows, fine_keys, ldf, pages, idx,
                       count, runs, run_count, (int)slots_cap);
  else
    hipLaunchKernelGGL((token_select_kernel<1024, true>), grid, dim3(1024), lds, st, g, n_rows, fine_keys, ldf, pages,
                       idx, count, runs, run_count, (int)slots_cap);
  return hipGetLastError();
}

__global__ __launch_bounds__(256) void fill_i32_kernel(int32_t* __restrict__ p, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

// Inverse of the run encoding: row r's runs [start, start + len) -> its position list
// idx[r, 0..count[r]) (cut at k_cap entries; lengths clamped to [0, k_cap], run counts to
// [0, k_cap]). One workgroup per row; thread t takes the contiguous block of runs
// [t U, t U + U), U = ceil(n_runs / 256), at the list offset a block prefix over the run
// lengths gives it, writes its short runs and queues the long ones (sink and window stretches),
// which the whole block then writes. Positions outside [0, 2^31) are written as -1 (skipped by
// attention).
__global__ __launch_bounds__(256) void expand_runs_kernel(const int32_t* __restrict__ runs,
                                                          const int32_t* __restrict__ run_count, int k_cap,
                                                          int32_t* __restrict__ idx, int32_t* __restrict__ count) {
  __shared__ int64_t wtot[4];
  const int64_t row = blockIdx.x;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int nr = run_count[row];
  nr = nr < 0 ? 0 : (nr > k_cap ? k_cap : nr);
  const int u = (nr + 255) / 256;
  const int b = (int)threadIdx.x * u < nr ? (int)threadIdx.x * u : nr;
  const int e = b + u < nr ? b + u : nr;
  const int32_t* rr = runs + row * k_cap * 2;
  auto len_of = [&](int r) {
    const int l = rr[2 * r + 1];
    return (int64_t)(l < 0 ? 0 : (l > k_cap ? k_cap : l));
  };
  int64_t mine = 0;
  for (int r = b; r < e; ++r) mine += len_of(r);
  int64_t inc = mine;  // inclusive prefix over the block
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t t = __shfl_up(inc, o);
    if (lane >= o) inc += t;
  }
  if (lane == 63) wtot[wv] = inc;
  __syncthreads();
  int64_t off = inc - mine, total = 0;
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    off += x < wv ? wtot[x] : 0;
    total += wtot[x];
  }
  // short runs are written by their thread; longer ones are queued and written by the whole block
  constexpr int kShort = 8, kQueue = 64;
  __shared__ int64_t qstart[kQueue];
  __shared__ int32_t qoff[kQueue], qlen[kQueue];
  __shared__ int qn;
  if (threadIdx.x == 0) qn = 0;
  __syncthreads();
  int32_t* out = idx + row * k_cap;
  auto put = [&](int64_t start, int64_t p0, int64_t n) {
    for (int64_t i = 0; i < n; ++i) {
      const int64_t v = start + i;
      out[p0 + i] = (v >= 0 && v < (1LL << 31)) ? (int32_t)v : -1;
    }
  };
  for (int r = b; r < e && off < k_cap; ++r) {
    const int64_t start = rr[2 * r], len = len_of(r);
    const int64_t n = (off + len < k_cap ? off + len : k_cap) - off;
    int slot = kQueue;
    if (n > kShort) slot = atomicAdd(&qn, 1);
    if (slot < kQueue) {
      qstart[slot] = start;
      qoff[slot] = (int32_t)off;
      qlen[slot] = (int32_t)n;
    } else {
      put(start, off, n);
    }
    off += len;
  }
  __syncthreads();
  const int nq = qn < kQueue ? qn : kQueue;
  for (int j = 0; j < nq; ++j)
    for (int i = (int)threadIdx.x; i < qlen[j]; i += 256) {
      const int64_t v = qstart[j] + i;
      out[qoff[j] + i] = (v >= 0 && v < (1LL << 31)) ? (int32_t)v : -1;
    }
  if (threadIdx.x == 0) count[row] = (int32_t)(total < k_cap ? total : k_cap);
}

hipError_t launch_expand_runs(const int32_t* runs, const int32_t* run_count, int64_t n_rows, int k_cap, int32_t* idx,
                              int32_t* count, hipStream_t st) {
  if (n_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(expand_runs_kernel, dim3((unsigned)n_rows), dim3(256), 0, st, runs, run_count, k_cap, idx, count);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_i32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

// Lets the two select kernels use up to 156 KB of dynamic LDS (gfx950 has 160 KB per
// workgroup); done once per device.
hipError_t prepare_index_kernels() {
  static std::atomic<bool> done[64] = {};  // per device; repeated setup by racing threads is harmless
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64 && done[dev].load(std::memory_order_acquire)) return hipSuccess;
  const int lim = (int)kSelectLdsLimit;
  const void* sel[] = {(const void*)token_select_kernel<512, false>, (const void*)token_select_kernel<1024, true>,
                       (const void*)token_select_reg_kernel<512, 16>, (const void*)token_select_reg_kernel<512, 32>,
                       (const void*)token_select_reg_kernel<512, 64>, (const void*)token_select_reg_kernel<1024, 8>};
  for (const void* f : sel) {  // (static LDS: under 4 KB in the first two, under 20 KB in the others)
    e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (f == sel[0] || f == sel[1]) ? lim : lim - 16 * 1024);
    if (e != hipSuccess) return e;
  }
  // the page selection's static LDS (range histograms) is under 8 KB
  e = hipFuncSetAttribute((const void*)page_select_kernel<256>, hipFuncAttributeMaxDynamicSharedMemorySize, lim - 4096);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute((const void*)page_select_kernel<1024>, hipFuncAttributeMaxDynamicSharedMemorySize, lim - 4096);
  if (e != hipSuccess) return e;

  if (dev >= 0 && dev < 64) done[dev].store(true, std::memory_order_release);
  return hipSuccess;
}

}  // namespace lsa
