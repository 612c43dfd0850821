// FP8 KV cache for long-context decode (paper section 2.3): per-tensor scale
// calibration at every RL step, quantised cache writes into a paged cache, and
// decode attention that reads the FP8 cache directly.
//
// Cache layout (one array each for K and V, one 2 KiB page per block and kv head):
//   K pages [num_blocks][kv_heads][16 tokens][128 dims] (token-major);
//   V pages [num_blocks][kv_heads][4][128 dims][4]: tokens 4a .. 4a+3 of each dim
//   are 4 adjacent bytes, so that the value product's MFMA operand (4 tokens of
//   8 dims per lane) is 32 contiguous bytes.
// token slot = block * 16 + offset; block_table [batch][max_blocks] int32.
//
// Decode attention ("KV cache FP8 only": the cache, not the arithmetic, is FP8):
//   scores:  E4M3 key codes widened exactly to bf16, times the bf16 query, by
//            v_mfma_f32_16x16x32_bf16 (16 tokens x 16 query-head columns, the
//            group's heads first), scaled by k_scale * sm_scale in fp32;
//   softmax: online per head in fp32;
//   values:  P (as a sum of two bf16 terms, 16 significant bits) x V (codes
//            widened exactly to bf16) by v_mfma_f32_16x16x16_bf16, 16 per page;
//            the score layout of the first product is already the P operand
//            layout of the second;
//   each wave covers one split of the sequence; a second kernel merges the
//   splits (log-sum-exp weights) and applies v_scale.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace fp8rl {
namespace {

constexpr int kDim = 128;          // head dimension
constexpr int kPage = 16;          // tokens per cache block
constexpr float kE4M3Max = 448.0f;

typedef __bf16 v8bf16_t __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf16_t __attribute__((ext_vector_type(2)));
typedef __bf16 v4bf16_t __attribute__((ext_vector_type(4)));
typedef float v4f32_t __attribute__((ext_vector_type(4)));
typedef float v2f32_t __attribute__((ext_vector_type(2)));

// ---------------------------------------------------------------------------
// Calibration: amax over a bf16 tensor (15-bit magnitude patterns order like the
// magnitudes), per-workgroup maxima into the workspace, then scale = amax / 448.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void amax_partial_kernel(const uint16_t* __restrict__ x, int64_t n,
                                                          uint32_t* __restrict__ partial) {
  __shared__ uint32_t red[4];
  uint32_t m = 0;
  const int64_t n8 = n / 8;
  const uint4* x8 = reinterpret_cast<const uint4*>(x);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n8; i += (int64_t)gridDim.x * 256)
    m = max(m, amax16_of(x8[i]));
  if (blockIdx.x == 0 && threadIdx.x < (n & 7)) m = max(m, (uint32_t)(x[n8 * 8 + threadIdx.x] & 0x7FFFu));
  m = wave_max(m);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) partial[blockIdx.x] = max(max(red[0], red[1]), max(red[2], red[3]));
}

__global__ __launch_bounds__(64) void scale_final_kernel(const uint32_t* __restrict__ partial, int blocks,
                                                        float* __restrict__ scale) {
  uint32_t m = 0;
  for (int b = threadIdx.x; b < blocks; b += 64) m = max(m, partial[b]);
  m = wave_max(m);
  if (threadIdx.x == 0) scale[0] = m == 0u ? 1.0f : __uint_as_float(m << 16) / kE4M3Max;   // IEEE division
}

// ---------------------------------------------------------------------------
// Cache write: one thread per (four consecutive tokens, kv head, 8-dim chunk)
// of K and V.  code = E4M3(fl32(x / s)) saturated at +-448 (IEEE division; the
// sign of x is OR-ed back so that -0 gives 0x80).  Slots outside
// [0, num_blocks * 16) are skipped (negative slots mark padding tokens).
// When the four tokens go to four consecutive slots starting at a multiple of 4
// (a prefill's tokens, in order), their value codes fill whole dwords of the
// value page (dim d: tokens 4a .. 4a+3) and are stored as 32 contiguous bytes;
// otherwise each token's value codes are stored byte by byte.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t quant4_static(uint32_t w0, uint32_t w1, float s) {
  float q[4] = {__uint_as_float(w0 << 16), __uint_as_float(w0 & 0xFFFF0000u), __uint_as_float(w1 << 16),
                __uint_as_float(w1 & 0xFFFF0000u)};
#pragma unroll
  for (int i = 0; i < 4; ++i) q[i] = fminf(fmaxf(q[i] / s, -kE4M3Max), kE4M3Max);
  int c = __builtin_amdgcn_cvt_pk_fp8_f32(q[0], q[1], 0, false);
  c = __builtin_amdgcn_cvt_pk_fp8_f32(q[2], q[3], c, true);
  const uint32_t signs = __builtin_amdgcn_perm(w1, w0, 0x07050301u) & 0x80808080u;
  return (uint32_t)c | signs;
}

// byte j of the result = byte `b` of word j (4x4 byte transpose, one output word)
__device__ __forceinline__ uint32_t gather_byte(const uint32_t (&w)[4], int b) {
  return ((w[0] >> (8 * b)) & 0xFFu) | (((w[1] >> (8 * b)) & 0xFFu) << 8) | (((w[2] >> (8 * b)) & 0xFFu) << 16) |
         (((w[3] >> (8 * b)) & 0xFFu) << 24);
}

__global__ __launch_bounds__(256) void kv_write_kernel(const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
                                                      int64_t tokens, int kv_heads, const int64_t* __restrict__ slots,
                                                      int64_t num_blocks, const float* __restrict__ k_scale,
                                                      const float* __restrict__ v_scale, uint8_t* __restrict__ kc,
                                                      uint8_t* __restrict__ vc) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per_quad = (int64_t)kv_heads * (kDim / 8);
  const int64_t quads = (tokens + 3) / 4;
  if (i >= quads * per_quad) return;
  const int64_t tq = i / per_quad;
  const int rem = (int)(i - tq * per_quad);
  const int h = rem / (kDim / 8), c = rem % (kDim / 8);
  const int64_t t0 = tq * 4;
  const int nt = (int)min((int64_t)4, tokens - t0);
  const int64_t limit = num_blocks * kPage;
  const float sk = k_scale[0], sv = v_scale[0];
  int64_t slot[4];
  uint32_t vlo[4] = {0u, 0u, 0u, 0u}, vhi[4] = {0u, 0u, 0u, 0u};   // value codes of dims c*8 .. +3, +4 .. +7
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    slot[r] = r < nt ? slots[t0 + r] : -1;
    if (r < nt) {
      const int64_t src = ((t0 + r) * kv_heads + h) * kDim + c * 8;
      const uint4 xk = *reinterpret_cast<const uint4*>(k + src);
      const uint4 xv = *reinterpret_cast<const uint4*>(v + src);
      vlo[r] = quant4_static(xv.x, xv.y, sv);
      vhi[r] = quant4_static(xv.z, xv.w, sv);
      if (slot[r] >= 0 && slot[r] < limit) {
        const int64_t blk = slot[r] / kPage, off = slot[r] % kPage;
        *reinterpret_cast<uint2*>(kc + ((blk * kv_heads + h) * kPage + off) * kDim + c * 8) =
            make_uint2(quant4_static(xk.x, xk.y, sk), quant4_static(xk.z, xk.w, sk));
      }
    }
  }
  const bool packed = nt == 4 && slot[0] >= 0 && slot[0] + 3 < limit && (slot[0] & 3) == 0 &&
                      slot[1] == slot[0] + 1 && slot[2] == slot[0] + 2 && slot[3] == slot[0] + 3;
  if (packed) {
    // dword of dim d = the four tokens' codes of d, dims c*8 .. c*8+7 contiguous
    const int64_t blk = slot[0] / kPage, off = slot[0] % kPage;
    uint4* vd = reinterpret_cast<uint4*>(vc + ((blk * kv_heads + h) * kPage * kDim) + ((off >> 2) * kDim + c * 8) * 4);
    vd[0] = make_uint4(gather_byte(vlo, 0), gather_byte(vlo, 1), gather_byte(vlo, 2), gather_byte(vlo, 3));
    vd[1] = make_uint4(gather_byte(vhi, 0), gather_byte(vhi, 1), gather_byte(vhi, 2), gather_byte(vhi, 3));
    return;
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (r >= nt || slot[r] < 0 || slot[r] >= limit) continue;
    // values: byte (off / 4, dim, off % 4) of the page
    const int64_t blk = slot[r] / kPage, off = slot[r] % kPage;
    uint8_t* vd = vc + (blk * kv_heads + h) * kPage * kDim + ((off >> 2) * kDim + c * 8) * 4 + (off & 3);
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      vd[4 * d] = (uint8_t)(vlo[r] >> (8 * d));
      vd[4 * (d + 4)] = (uint8_t)(vhi[r] >> (8 * d));
    }
  }
}

// ---------------------------------------------------------------------------
// Decode attention.
// ---------------------------------------------------------------------------
template <bool kFp8>
struct CacheElem;
template <>
struct CacheElem<true> { typedef uint8_t T; };
template <>
struct CacheElem<false> { typedef uint16_t T; };

typedef short v4i16_t __attribute__((ext_vector_type(4)));

// 8 consecutive cache values -> 8 bf16 (exact: every E4M3 value is a bf16 value)
__device__ __forceinline__ v8bf16_t to_bf16x8(const uint2& c) {
  const v2bf16_t a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)c.x, 1.0f, false);
  const v2bf16_t b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)c.x, 1.0f, true);
  const v2bf16_t d = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)c.y, 1.0f, false);
  const v2bf16_t e = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)c.y, 1.0f, true);
  return (v8bf16_t){a[0], a[1], b[0], b[1], d[0], d[1], e[0], e[1]};
}
__device__ __forceinline__ v8bf16_t to_bf16x8(const uint4& c) { return __builtin_bit_cast(v8bf16_t, c); }

// 4 consecutive cache values -> 4 bf16 as the 16x16x16 MFMA operand
__device__ __forceinline__ v4i16_t to_bf16x4(uint32_t c) {
  const v2bf16_t a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)c, 1.0f, false);
  const v2bf16_t b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)c, 1.0f, true);
  return __builtin_bit_cast(v4i16_t, (v4bf16_t){a[0], a[1], b[0], b[1]});
}
__device__ __forceinline__ v4i16_t to_bf16x4(const uint2& c) { return __builtin_bit_cast(v4i16_t, c); }

// Per lane and page: keys = 32 contiguous cache values (token L % 16, dims 32 (L / 16) ..),
// values = 32 contiguous cache values (tokens 4 (L / 16) .. +3 of dims 8 (L % 16) .. +7).
template <bool kFp8>
struct PageRegs;
template <>
struct PageRegs<true> {
  uint4 k[2];
  uint4 v[2];
};
template <>
struct PageRegs<false> {
  uint4 k[4];
  uint4 v[4];
};

__device__ __forceinline__ float shfl_xor_f(float v, int m) { return __shfl_xor(v, m, 64); }

// Partial record per (sequence, kv head, split): o[G][128], then m[G], l[G],
// padded to a multiple of 4 floats (16-byte aligned records).
template <int kG>
constexpr int partial_floats() { return kG * kDim + (2 * kG + 3) / 4 * 4; }
template <int kG>
constexpr int rec_m() { return kG * kDim; }
template <int kG>
constexpr int rec_l() { return kG * kDim + kG; }

// Workgroup = 4 waves = 4 consecutive splits of one (sequence, kv head); wave w
// covers tokens [split * split_tokens, +split_tokens) of the sequence.  Lane L,
// g = L / 16, j = L % 16:
//   score product (16x16x32, 4 per page): A = keys of token j, dims 32g + 8kk ..
//     (the same dim permutation for the query operand, column j = head j of the
//     group, zero past kG); the result holds S[token 4g + i][head j];
//   online softmax per head j (lanes j hold head j's running max and sum);
//   value product (16x16x16, 8 per page, nb = 0..7): A = P[head j][tokens 4g ..
//     4g+3] (exactly the score layout), B = V[tokens 4g .. 4g+3][dim 8j + nb];
//     the result holds O[head 4g + i][dim 8j + nb].
template <int kG, bool kFp8>
__global__ __launch_bounds__(256) void attn_decode_kernel(
    const uint16_t* __restrict__ q, const typename CacheElem<kFp8>::T* __restrict__ kcache,
    const typename CacheElem<kFp8>::T* __restrict__ vcache, int64_t num_blocks,
    const int32_t* __restrict__ block_table, int max_blocks, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ k_scale, float sm_scale, int kv_heads, int split_tokens, int max_splits,
    float* __restrict__ partial) {
  typedef typename CacheElem<kFp8>::T E;
  constexpr int kPer16 = 16 / sizeof(E);                  // cache values per 16-byte load
  const int lane = threadIdx.x & 63;
  // wave-uniform as far as the compiler knows too: the split, its token range and
  // the page indices stay in scalar registers, so the block-table reads are scalar
  // loads (a vector load there would make each page's loads wait for every load in
  // flight, the prefetched pages included)
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int split = blockIdx.x * 4 + wave;
  if (split >= max_splits) return;
  const int kvh = blockIdx.y;
  const int b = blockIdx.z;
  const int g = lane >> 4, j = lane & 15;
  const int n = seq_lens[b];
  const int t0 = split * split_tokens;
  const int t1 = min(n, t0 + split_tokens);
  float* rec = partial + (((int64_t)b * kv_heads + kvh) * max_splits + split) * partial_floats<kG>();

  // query operand: head j of the group (zero columns past kG), dims 32g + 8kk ..+7
  v8bf16_t qb[4];
  {
    const int head = kvh * kG + min(j, kG - 1);
    const uint16_t* qrow = q + ((int64_t)b * kv_heads * kG + head) * kDim + 32 * g;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const uint4 w = *reinterpret_cast<const uint4*>(qrow + 8 * kk);
      qb[kk] = __builtin_bit_cast(v8bf16_t, j < kG ? w : make_uint4(0u, 0u, 0u, 0u));
    }
  }
  const float sscale = (k_scale ? k_scale[0] : 1.0f) * sm_scale;     // bf16 cache: no scale
  float m = -INFINITY, l = 0.0f;                 // running max / sum of head j
  v4f32_t o[8];
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) o[nb] = (v4f32_t){0.f, 0.f, 0.f, 0.f};

  const int64_t head_stride = (int64_t)kPage * kDim;            // one kv head's page
  auto load_page = [&](int tp, PageRegs<kFp8>& r) {
    const int page = min(tp / kPage, max_blocks - 1);
    int64_t blk = block_table[(int64_t)b * max_blocks + page];
    blk = blk < 0 ? 0 : (blk >= num_blocks ? num_blocks - 1 : blk);   // a bad entry reads a wrong page, never outside
    const int64_t base = (blk * kv_heads + kvh) * head_stride;
    const E* kp = kcache + base + j * kDim + 32 * g;
    const E* vp = vcache + base + (g * kDim + 8 * j) * 4;
#pragma unroll
    for (int c = 0; c < 32 / kPer16; ++c) {
      r.k[c] = *reinterpret_cast<const uint4*>(kp + c * kPer16);
      r.v[c] = *reinterpret_cast<const uint4*>(vp + c * kPer16);
    }
  };

  // Three pages in flight: the current one and the next two, in three register
  // sets that rotate by name (the loop body below runs three pages), so no page's
  // registers are copied while a later page's loads into them are in flight.
  // Every step issues its prefetch unconditionally (past the split's end it
  // re-reads the split's last page, a cache hit): with the same number of loads
  // on every path the compiler waits for exactly the page it needs, never for
  // the prefetches behind it.
  if (t0 >= t1) return;    // (empty split: nothing in flight, nothing to write)
  const int t_last = t1 - 1;
  PageRegs<kFp8> pg0, pg1, pg2;
  load_page(t0, pg0);
  load_page(min(t0 + kPage, t_last), pg1);
  // one page: prefetch page tp + 2 into `next` (the set of page tp - 1), then
  // attend over page tp held in `cur` if it is inside the split
  auto page_step = [&](int tp, const PageRegs<kFp8>& cur, PageRegs<kFp8>& next) {
    load_page(min(tp + 2 * kPage, t_last), next);
    if (tp >= t1) return;
    const int valid = min(kPage, t1 - tp);

    // ---- scores
    v4f32_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      v8bf16_t a;
      if constexpr (kFp8) {
        const uint4& w = cur.k[kk >> 1];
        a = to_bf16x8((kk & 1) ? make_uint2(w.z, w.w) : make_uint2(w.x, w.y));
      } else {
        a = to_bf16x8(cur.k[kk]);
      }
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qb[kk], acc, 0, 0, 0);
    }
    // ---- online softmax for head j (tokens 4g + i of the page)
    float s[4], mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s[i] = (4 * g + i < valid) ? acc[i] * sscale : -INFINITY;
      mx = fmaxf(mx, s[i]);
    }
    mx = fmaxf(mx, shfl_xor_f(mx, 16));
    mx = fmaxf(mx, shfl_xor_f(mx, 32));
    const float m_new = fmaxf(m, mx);                       // finite: the page has a valid token
    const float alpha = __expf(m - m_new);                  // 0 on the first page
    float psum = 0.0f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      s[i] = __expf(s[i] - m_new);                          // masked tokens: 0
      psum += s[i];
    }
    psum += shfl_xor_f(psum, 16);
    psum += shfl_xor_f(psum, 32);
    l = l * alpha + psum;
    m = m_new;
    // rows of o are heads 4g + i: rescale by their alphas (held by lanes 4g + i)
    if (__ballot(j < kG && alpha != 1.0f)) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float ai = __shfl(alpha, 4 * g + i, 64);
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) o[nb][i] *= ai;
      }
    }
    // ---- values: P[head j][tokens 4g .. 4g+3] in bf16 (masked tokens are 0); the
    //      values of tokens past the sequence end are zeroed too (unwritten cache
    //      bytes may hold NaN codes, and 0 x NaN is NaN)
    // P as the sum of two bf16 terms (16 significant bits; one bf16 term alone
    // leaves errors of 2^-9 of each weight), two MFMAs per value tile
    const v4bf16_t p_hi = {(__bf16)s[0], (__bf16)s[1], (__bf16)s[2], (__bf16)s[3]};
    const v4bf16_t p_lo = {(__bf16)(s[0] - (float)p_hi[0]), (__bf16)(s[1] - (float)p_hi[1]),
                           (__bf16)(s[2] - (float)p_hi[2]), (__bf16)(s[3] - (float)p_hi[3])};
    const v4i16_t pa = __builtin_bit_cast(v4i16_t, p_hi), pb = __builtin_bit_cast(v4i16_t, p_lo);
    const int keep = min(max(valid - 4 * g, 0), 4);                  // tokens of this lane's four
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) {
      v4i16_t vb;
      if constexpr (kFp8) {
        const uint4& w = cur.v[nb >> 2];
        uint32_t word = (nb & 3) == 0 ? w.x : (nb & 3) == 1 ? w.y : (nb & 3) == 2 ? w.z : w.w;
        word &= keep >= 4 ? 0xFFFFFFFFu : (1u << (8 * keep)) - 1u;
        vb = to_bf16x4(word);
      } else {
        const uint4& w = cur.v[nb >> 1];
        uint2 pr = (nb & 1) ? make_uint2(w.z, w.w) : make_uint2(w.x, w.y);
        pr.x &= keep >= 2 ? 0xFFFFFFFFu : (keep == 1 ? 0xFFFFu : 0u);
        pr.y &= keep >= 4 ? 0xFFFFFFFFu : (keep == 3 ? 0xFFFFu : 0u);
        vb = to_bf16x4(pr);
      }
      o[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa, vb, o[nb], 0, 0, 0);
      o[nb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pb, vb, o[nb], 0, 0, 0);
    }
  };
  for (int tp = t0; tp < t1; tp += 3 * kPage) {
    page_step(tp, pg0, pg2);
    page_step(tp + kPage, pg1, pg0);
    page_step(tp + 2 * kPage, pg2, pg1);
  }

  // o[nb][i] = O[head 4g + i][dim 8j + nb]; lanes h < kG of group 0 hold m, l of head h
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int head = 4 * g + i;
    if (head < kG) {
      float4* dst = reinterpret_cast<float4*>(rec + head * kDim + 8 * j);
      dst[0] = make_float4(o[0][i], o[1][i], o[2][i], o[3][i]);
      dst[1] = make_float4(o[4][i], o[5][i], o[6][i], o[7][i]);
    }
  }
  if (g == 0 && j < kG) {
    rec[rec_m<kG>() + j] = m;
    rec[rec_l<kG>() + j] = l;
  }
}

// out[b][head][d] = bf16( v_scale * sum_s e^(m_s - M) o_s[d] / sum_s e^(m_s - M) l_s ),
// one workgroup of 64 threads (two dims each) per (head, sequence); empty
// sequences give 0.
template <int kG>
__global__ __launch_bounds__(64) void attn_merge_kernel(const float* __restrict__ partial,
                                                       const int32_t* __restrict__ seq_lens,
                                                       const float* __restrict__ v_scale, int kv_heads,
                                                       int split_tokens, int max_splits, uint16_t* __restrict__ out) {
  const int head = blockIdx.x, b = blockIdx.y;
  const int kvh = head / kG, h = head % kG;
  const int n = seq_lens[b];
  const int ns = min(max_splits, (max(n, 0) + split_tokens - 1) / split_tokens);
  const float* base = partial + ((int64_t)b * kv_heads + kvh) * max_splits * partial_floats<kG>();
  float mmax = -INFINITY;
  for (int s = 0; s < ns; ++s) mmax = fmaxf(mmax, base[(int64_t)s * partial_floats<kG>() + rec_m<kG>() + h]);
  float lsum = 0.0f, a0 = 0.0f, a1 = 0.0f;
  const int d = 2 * threadIdx.x;
  for (int s = 0; s < ns; ++s) {
    const float* r = base + (int64_t)s * partial_floats<kG>();
    const float w = expf(r[rec_m<kG>() + h] - mmax);
    lsum += r[rec_l<kG>() + h] * w;
    a0 += r[h * kDim + d] * w;
    a1 += r[h * kDim + d + 1] * w;
  }
  const float f = ns > 0 ? (v_scale ? v_scale[0] : 1.0f) / lsum : 0.0f;
  const uint32_t o2 = f32_to_bf16_rne(a0 * f) | (f32_to_bf16_rne(a1 * f) << 16);
  *reinterpret_cast<uint32_t*>(out + ((int64_t)b * kv_heads * kG + head) * kDim + d) = o2;
}

}  // namespace

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
int kv_amax_blocks(int64_t n) {
  const int64_t b = (n / 8 + 255) / 256;
  return (int)(b < 1 ? 1 : (b > 1024 ? 1024 : b));
}

hipError_t launch_kv_calibrate_scale(const uint16_t* x, int64_t n, float* scale, uint32_t* partial,
                                     hipStream_t stream) {
  const int blocks = kv_amax_blocks(n);
  hipLaunchKernelGGL(amax_partial_kernel, dim3(blocks), dim3(256), 0, stream, x, n, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(scale_final_kernel, dim3(1), dim3(64), 0, stream, partial, blocks, scale);
  return hipGetLastError();
}

hipError_t launch_kv_cache_write(const uint16_t* k, const uint16_t* v, int64_t tokens, int kv_heads,
                                 const int64_t* slots, int64_t num_blocks, const float* k_scale, const float* v_scale,
                                 uint8_t* k_cache, uint8_t* v_cache, hipStream_t stream) {
  const int64_t threads = (tokens + 3) / 4 * kv_heads * (kDim / 8);
  hipLaunchKernelGGL(kv_write_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream, k, v, tokens,
                     kv_heads, slots, num_blocks, k_scale, v_scale, k_cache, v_cache);
  return hipGetLastError();
}

AttnSplit attn_decode_split(int64_t batch, int64_t kv_heads, int64_t group, int64_t max_seq_len) {
  // about 6144 waves over the whole batch (three times the 2048 that are resident
  // at two waves per SIMD), splits of at least 256 tokens.  Measured on 64
  // sequences of 4096 .. 20480 tokens: 2048 / 3072 / 4096 / 6144 / 8192 / 16384
  // waves took 396 / 440 / 385 / 358 / 394 / 429 us.
  constexpr int64_t kTargetWaves = 6144;
  const int64_t pairs = batch * kv_heads;
  int64_t splits = (kTargetWaves + pairs - 1) / (pairs > 0 ? pairs : 1);
  if (splits < 1) splits = 1;
  int64_t per = (max_seq_len + splits - 1) / splits;
  per = (per + kPage - 1) / kPage * kPage;
  if (per < 256) per = 256;
  AttnSplit s;
  s.split_tokens = (int)per;
  s.max_splits = (int)((max_seq_len + per - 1) / per);
  if (s.max_splits < 1) s.max_splits = 1;
  s.partial_floats = (int)(group * kDim + (2 * group + 3) / 4 * 4);   // as partial_floats<G>()
  return s;
}

template <int kG, bool kFp8>
static hipError_t launch_attn(const uint16_t* q, const void* kc, const void* vc, int64_t num_blocks,
                              const int32_t* block_table, int64_t max_blocks, const int32_t* seq_lens, int64_t batch,
                              int64_t kv_heads, const AttnSplit& sp, const float* k_scale, const float* v_scale,
                              float sm_scale, uint16_t* out, float* partial, hipStream_t stream) {
  typedef typename CacheElem<kFp8>::T E;
  dim3 grid((unsigned)((sp.max_splits + 3) / 4), (unsigned)kv_heads, (unsigned)batch);
  hipLaunchKernelGGL((attn_decode_kernel<kG, kFp8>), grid, dim3(256), 0, stream, q, static_cast<const E*>(kc),
                     static_cast<const E*>(vc), num_blocks, block_table, (int)max_blocks, seq_lens, k_scale, sm_scale,
                     (int)kv_heads, sp.split_tokens, sp.max_splits, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_merge_kernel<kG>), dim3((unsigned)(kv_heads * kG), (unsigned)batch), dim3(64), 0, stream,
                     partial, seq_lens, v_scale, (int)kv_heads, sp.split_tokens, sp.max_splits, out);
  return hipGetLastError();
}

hipError_t launch_attention_decode(const uint16_t* q, const void* k_cache, const void* v_cache, bool fp8_cache,
                                   int64_t num_blocks, const int32_t* block_table, int64_t max_blocks,
                                   const int32_t* seq_lens, int64_t batch, int64_t q_heads, int64_t kv_heads,
                                   int64_t max_seq_len, const float* k_scale, const float* v_scale, float sm_scale,
                                   uint16_t* out, float* partial, hipStream_t stream) {
  const int64_t group = q_heads / kv_heads;
  const AttnSplit sp = attn_decode_split(batch, kv_heads, group, max_seq_len);
#define FP8RL_ATTN(G)                                                                                            \
  if (group == G)                                                                                                \
    return fp8_cache ? launch_attn<G, true>(q, k_cache, v_cache, num_blocks, block_table, max_blocks, seq_lens,  \
                                            batch, kv_heads, sp, k_scale, v_scale, sm_scale, out, partial, stream) \
                     : launch_attn<G, false>(q, k_cache, v_cache, num_blocks, block_table, max_blocks, seq_lens, \
                                             batch, kv_heads, sp, k_scale, v_scale, sm_scale, out, partial, stream);
  FP8RL_ATTN(1)
  FP8RL_ATTN(2)
  FP8RL_ATTN(4)
  FP8RL_ATTN(8)
#undef FP8RL_ATTN
  return hipErrorInvalidValue;
}

}  // namespace fp8rl
