// Sparse attention over an index list (Eq. 3 of "LongCat Sparse Attention", arXiv 2608.01662)
// for gfx950: MLA absorbed mode (64 heads, latent rows of 576 = 512 + 64 bf16, V = first 512
// columns) and MQA-128 (16 heads, separate K and V of 128).
//
// Both kernels compute S^T = K Q^T (keys on the MFMA rows, heads on the columns) so that in the
// accumulator layout each lane holds 16 (or 8) tokens of ONE head: the per-head softmax max and
// sum are in-lane reductions plus one or two lane exchanges, and the exponentiated scores are
// already in the B-operand layout of the next product O^T += V^T P^T. V^T reaches the A-operand
// layout through ds_read_b64_tr_b16 (a 16 x 4 transpose read on gfx950), so V is stored once,
// token-major, in the same LDS tile as K.
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

// acc *= alpha on an MFMA accumulator kept in AGPRs, element by element through one VGPR. Written
// as asm so that the accumulators never need VGPR copies outside this (rare) path.
__device__ __forceinline__ f32x16 scale_acc(f32x16 acc, float alpha) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float x = acc[r], t;
    asm volatile("v_accvgpr_read_b32 %1, %0\n\tv_mul_f32 %1, %1, %2\n\tv_accvgpr_write_b32 %0, %1"
                 : "+a"(x), "=&v"(t)
                 : "v"(alpha));
    acc[r] = x;
  }
  return acc;
}

__device__ __forceinline__ u32x4 tr16_pair(const uint8_t* pa, const uint8_t* pb) {
  const s16x4 va = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(pa));
  const s16x4 vb = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(pb));
  const u32x2 a2 = __builtin_bit_cast(u32x2, va), b2 = __builtin_bit_cast(u32x2, vb);
  return u32x4{a2.x, a2.y, b2.x, b2.y};
}

// ============================================================================ MLA 64 x 576 / 512
// One workgroup = 4 waves = one query row (or one split of it). Wave (hw, kw) = (w >> 1, w & 1)
// owns heads 32hw..32hw+31 and
//   * computes the partial S^T over dims [288 kw, 288 kw + 288) of the 576 (18 MFMA k-steps);
//     the two partials of a head half are summed through a 16 KB LDS exchange,
//   * accumulates O^T for value columns [256 kw, 256 kw + 256) (8 tiles of 32 x 32).
// Every wave does the same MFMA work and holds 72 Q-operand and 128 accumulator registers.
//
// KV tiles of 32 gathered latent rows are double-buffered in LDS by direct global->LDS loads
// (no VGPR staging). LDS tile layout is chunk-major: 16-byte chunk c (dims 8c..8c+7) of token t
// sits at c*512 + (t ^ 4*(c&1))*16. Each direct load moves chunks (2k, 2k+1) of all 32 tokens,
// so a lane reads one token row at base + 32k and the lines of a row are fetched by consecutive
// instructions; the K-operand reads are 512 contiguous bytes per half-wave.
constexpr int kMlaT = 32;
constexpr int kMlaLoads = 9;              // direct loads per wave per tile (36 per tile)
constexpr int kMlaBuf = 36 * 1024;        // 36864 bytes per tile buffer
constexpr int kMlaXch = 4 * 4096;         // partial-score exchange, 4 KB per wave

template <bool SPLIT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void mla_attn_kernel(AttnGeom a) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * kMlaBuf + kMlaXch];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, h = lane >> 5, j = lane & 31;
  const int hw = wv >> 1, kw = wv & 1;
  const int64_t row = xcd_band(blockIdx.x, a.n_rows);
  const int split = SPLIT ? (int)blockIdx.y : 0;
  int cnt = a.count[row];
  cnt = cnt < 0 ? 0 : (cnt > a.k_cap ? a.k_cap : cnt);
  const int s0 = split * a.split_len;
  const int s1 = SPLIT ? (cnt < s0 + a.split_len ? cnt : s0 + a.split_len) : cnt;
  const int n = s1 > s0 ? s1 - s0 : 0;
  const int ntiles = (n + kMlaT - 1) / kMlaT;
  const int32_t* slots = a.rows + row * a.k_cap + s0;
  const uint8_t* kvb = reinterpret_cast<const uint8_t*>(a.kv);
  const int head = 32 * hw + j;
  uint8_t* xch = lds + 2 * kMlaBuf;

  // Q^T as the B operand of S^T = K Q^T: column = head, k-step s covers dims 16s + 8h .. +7,
  // s in [18 kw, 18 kw + 18).
  u32x4 qb[18];
  {
    const u32x4* qp = reinterpret_cast<const u32x4*>(a.q + (row * 64 + head) * 576 + 8 * h) + 36 * kw;
#pragma unroll
    for (int s = 0; s < 18; ++s) qb[s] = qp[2 * s];
  }
  f32x16 o[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) o[c] = f32x16{};
  float m = -INFINITY, l = 0.f;

  auto fetch = [&](int tile) -> int {  // exactly one load per call
    const int sl = tile * kMlaT + j;
    return slots[sl < n ? sl : n - 1];
  };
  auto checked = [&](int tile, int r) -> int {
    const int sl = tile * kMlaT + j;
    return (sl < n && r >= 0 && (int64_t)r < a.n_kv_rows) ? r : -1;
  };
  // direct load K = 9w + k moves chunks (2K, 2K+1); lane (j, h) fills slot j of chunk 2K + h,
  // which holds token j ^ 4h ^ 8(K&1).
  auto issue = [&](int prow, int buf) {
    const int pr = __shfl(prow, j ^ (4 * h));
    const uint8_t* src = kvb + (pr >= 0 ? (int64_t)pr * 1152 : 0) + 16 * h + 32 * (wv * kMlaLoads);
    uint8_t* dst = lds + buf * kMlaBuf + wv * (kMlaLoads * 1024);
#pragma unroll
    for (int k = 0; k < kMlaLoads; ++k)
      __builtin_amdgcn_global_load_lds(src + 32 * k, LSA_LDS(dst + k * 1024), 16, 0, 0);
  };

  if (ntiles > 0) {
    const int raw0 = fetch(0);
    int raw_next = fetch(ntiles > 1 ? 1 : 0);
    int r_cur = checked(0, raw0);
    issue(r_cur, 0);
    for (int it = 0; it < ntiles; ++it) {
      int r_next = -1;
      if (it + 1 < ntiles) {
        r_next = checked(it + 1, raw_next);
        issue(r_next, (it + 1) & 1);
        raw_next = fetch(it + 2 < ntiles ? it + 2 : it + 1);
        vm_wait_barrier<kMlaLoads + 1>();
      } else {
        vm_wait_barrier<0>();
      }
      const uint8_t* tb = lds + (it & 1) * kMlaBuf;

      // ---- partial S^T = K Q^T over this wave's 288 dims; K operand: token j, chunk 2s + h
      f32x16 sacc = {};
      // K operand: token j, chunk c = 36kw + 2s + h, slot j ^ 4h ^ 8((c>>1)&1), (c>>1)&1 = (18kw+s)&1
      const uint8_t* kp = tb + (36 * kw + h) * 512 + (j ^ (4 * h)) * 16;
#pragma unroll
      for (int s = 0; s < 18; ++s) {
        const u32x4 ka = *reinterpret_cast<const u32x4*>(kp + s * 1024);
        sacc = mfma32(ka, qb[s], sacc);
      }
      // ---- sum the two partials of this head half through LDS
      {
        f32x4* mine = reinterpret_cast<f32x4*>(xch + wv * 4096) + lane;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) mine[64 * q4] = f32x4{sacc[4 * q4], sacc[4 * q4 + 1], sacc[4 * q4 + 2], sacc[4 * q4 + 3]};
        lds_done_barrier();
        const f32x4* other = reinterpret_cast<const f32x4*>(xch + (wv ^ 1) * 4096) + lane;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const f32x4 v = other[64 * q4];
          sacc[4 * q4] += v[0]; sacc[4 * q4 + 1] += v[1]; sacc[4 * q4 + 2] += v[2]; sacc[4 * q4 + 3] += v[3];
        }
      }
      // ---- online softmax (base 2); lane holds tokens 8(r/4) + 4h + r%4 of head `head`.
      // Both waves of a head half see the same sums in the same order, so they agree exactly.
      const uint32_t vmask = (uint32_t)__ballot(r_cur >= 0);
      if (vmask != 0xFFFFFFFFu) {  // partial or invalid tokens (last tile of a row): mask them
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int tk = 8 * (r / 4) + 4 * h + (r % 4);
          sacc[r] = ((vmask >> tk) & 1u) ? sacc[r] : -INFINITY;
        }
      }
      float smax = sacc[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) smax = fmaxf(smax, sacc[r]);
      smax = fmaxf(smax, __shfl_xor(smax, 32));
      const float mx = smax * a.scale_log2;  // scale > 0: max commutes with scaling
      const bool need = mx > m + kLazy;
      if (__ballot(need)) {
        // Rare after the first tile (the reference max only moves by > 2^8). The asm keeps the
        // compiler from turning this branch into an every-tile multiply of all accumulators.
        const float alpha = need ? fast_exp2(m - mx) : 1.f;
#pragma unroll
        for (int c = 0; c < 8; ++c) o[c] = scale_acc(o[c], alpha);
        l *= alpha;
        m = need ? mx : m;
      }
      const float mb = m == -INFINITY ? 0.f : m;  // m = -inf only while every score is -inf
      float p[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        p[r] = fast_exp2(fmaf(sacc[r], a.scale_log2, -mb));  // -inf -> 0
        l += p[r];
      }
      const u32x4 pb0 = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3]), pack_bf16x2(p[4], p[5]), pack_bf16x2(p[6], p[7])};
      const u32x4 pb1 = {pack_bf16x2(p[8], p[9]), pack_bf16x2(p[10], p[11]), pack_bf16x2(p[12], p[13]),
                         pack_bf16x2(p[14], p[15])};
      // ---- O^T += V^T P^T over this wave's 256 value columns; V^T via transposed LDS reads.
      // 16-lane group (column half ch16 = (lane>>4)&1, token half h); source lane (vq, gq) reads
      // token t0 + vq, dims 32c + 16*ch16 + 4gq .. +3, i.e. chunk 4c + 2*ch16 + gq/2.
      const int gi = lane & 15, vq = gi >> 2, gq = gi & 3;
      const int ch16 = (lane >> 4) & 1;
      // chunk 32kw + 4c + 2ch16 + gq/2: (c&1) = gq/2, ((c>>1)&1) = ch16
      const int sw = 4 * (gq >> 1);
      const uint8_t* vb = tb + (32 * kw + 2 * ch16 + (gq >> 1)) * 512 + (gq & 1) * 8;
      const int t0 = 4 * h + vq;
      const int oa = (t0 ^ sw) * 16, ob = ((t0 + 8) ^ sw) * 16, oc = ((t0 + 16) ^ sw) * 16, od = ((t0 + 24) ^ sw) * 16;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const uint8_t* pc = vb + c * 2048;
        o[c] = mfma32(tr16_pair(pc + oa, pc + ob), pb0, o[c]);
        o[c] = mfma32(tr16_pair(pc + oc, pc + od), pb1, o[c]);
      }
      lds_done_barrier();  // tile buffer and exchange slots are free again
      r_cur = r_next;
    }
  }

  const float lt = l + __shfl_xor(l, 32);
  const int dv0 = 256 * kw + 4 * h;
  if (!SPLIT) {
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    uint16_t* orow = a.out + (row * 64 + head) * 512 + dv0;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const u32x2 v = {pack_bf16x2(o[c][4 * rr] * inv, o[c][4 * rr + 1] * inv),
                         pack_bf16x2(o[c][4 * rr + 2] * inv, o[c][4 * rr + 3] * inv)};
        *reinterpret_cast<u32x2*>(orow + 32 * c + 8 * rr) = v;
      }
    }
    if (a.lse && h == 0 && kw == 0) a.lse[row * 64 + head] = lt > 0.f ? (m + __log2f(lt)) * kLn2 : -INFINITY;
  } else {
    const int64_t pi = (row * a.n_split + split) * 64 + head;
    float* po = a.part_o + pi * 512 + dv0;
#pragma unroll
    for (int c = 0; c < 8; ++c) {
#pragma unroll
      for (int rr = 0; rr < 4; ++rr)
        *reinterpret_cast<f32x4*>(po + 32 * c + 8 * rr) =
            f32x4{o[c][4 * rr], o[c][4 * rr + 1], o[c][4 * rr + 2], o[c][4 * rr + 3]};
    }
    if (h == 0 && kw == 0) {
      a.part_ml[pi * 2] = m;
      a.part_ml[pi * 2 + 1] = lt;
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
// merge partial attentions, Sec. 4.1.1 and App. B). Grid (n_rows, H), block 128.
__global__ __launch_bounds__(128) void attn_combine_kernel(AttnGeom a, int H, int d_v) {
  const int64_t row = blockIdx.x;
  const int head = blockIdx.y;
  float M = -INFINITY;
  for (int s = 0; s < a.n_split; ++s) M = fmaxf(M, a.part_ml[((row * a.n_split + s) * H + head) * 2]);
  float L = 0.f;
  for (int s = 0; s < a.n_split; ++s) {
    const int64_t pi = (row * a.n_split + s) * H + head;
    const float ms = a.part_ml[pi * 2], ls = a.part_ml[pi * 2 + 1];
    L += ls > 0.f ? ls * fast_exp2(ms - M) : 0.f;
  }
  const float inv = L > 0.f ? 1.f / L : 0.f;
  for (int d = threadIdx.x * 4; d < d_v; d += 128 * 4) {
    f32x4 acc = {};
    for (int s = 0; s < a.n_split; ++s) {
      const int64_t pi = (row * a.n_split + s) * H + head;
      const float ls = a.part_ml[pi * 2 + 1];
      if (!(ls > 0.f)) continue;
      const float wgt = fast_exp2(a.part_ml[pi * 2] - M);
      acc += wgt * *reinterpret_cast<const f32x4*>(a.part_o + pi * d_v + d);
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
hipError_t launch_mla_attn(const AttnGeom& a, hipStream_t st) {
  if (a.n_rows == 0) return hipSuccess;
  if (a.n_split > 1) {
    hipLaunchKernelGGL(mla_attn_kernel<true>, dim3((unsigned)a.n_rows, (unsigned)a.n_split), dim3(256), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_attn_combine(a, 64, 512, st);
  }
  hipLaunchKernelGGL(mla_attn_kernel<false>, dim3((unsigned)a.n_rows), dim3(256), 0, st, a);
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

hipError_t prepare_attn_kernels() { return hipSuccess; }

}  // namespace lsa
