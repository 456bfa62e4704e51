// Device half of libq4nx for gfx950: the Q4NX dequantization kernel
// (Sec. 3.1.1), the fused dequant mat-vec of the decode phase (FusedDQP,
// Sec. 3.2.1, Eq. 14/15) and the fused dequant matrix product of the prefill
// phase (Sec. 3.1.2), with their C-ABI launchers -- for Q4NX blocks and for
// the MXFP4 variant of the block (FP4 E2M1 codes, one E8M0 scale per group).
//
// Common lane mapping inside a 32 x 256 block: a 16-byte load by lane l at
// byte 1024t + 16l of the block holds the 32 codes of one quantization group,
// row r = 8t + l/8, group c = l%8 (columns 32c..32c+31).  So a wave reads a
// whole block with four fully coalesced 1 KiB loads, and the scale/offset of
// the lane's group sits at index 8r + c = 64t + l of the block's tables.
#include <hip/hip_runtime.h>

#include <cstdlib>
#include <string>
#include <vector>

#include "q4nx_device.h"
#include "q4nx_internal.h"
#include "q4nx_xlane.h"

namespace q4nx {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------

// Hides the known bits of a value from the optimizer, so that byte extraction
// of a masked word maps onto v_cvt_f32_ubyte{0..3} (one op per code) instead
// of a per-code AND followed by a convert.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 p = __builtin_convertvector((float __attribute__((ext_vector_type(2)))){a, b}, bf16x2);
  return __builtin_bit_cast(uint32_t, p);
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float a) {
  return (uint16_t)(pack_bf16x2(a, 0.0f) & 0xFFFFu);
}

// Streaming loads of the packed weights (read once per call).
__device__ __forceinline__ u32x4 load_codes(const uint8_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ uint32_t load_u16(const uint8_t* p) {
  return (uint32_t)__builtin_nontemporal_load(reinterpret_cast<const uint16_t*>(p));
}

// A byte holding a 4-bit code q, read as an FP8 E4M3 value, is exactly
// q * 2^-9 (codes 0..7 are the subnormals m * 2^-9, codes 8..15 the first
// normal binade (8 + m) * 2^-9), so one gfx950 conversion turns two code bytes
// into two exact bf16 values; the conversion's scale operand 2^9 makes them q.
template <bool HI_WORD>
__device__ __forceinline__ bf16x2 codes2_bf16(uint32_t bytes) {
  return __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(bytes, 512.0f, HI_WORD);
}

// sum_i q_i * x_i over one group of 32 codes (one 16-byte word), with x given
// as 16 bf16 pairs in the order the nibble split produces: for each 8-column
// run u, (x0,x2), (x4,x6), (x1,x3), (x5,x7).  Products of two bf16 values are
// exact; v_dot2 adds two of them to the float32 accumulator.
__device__ __forceinline__ float group_dot_bf16(u32x4 q, const uint32_t (&xp)[16]) {
  float a = 0.0f, b = 0.0f;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const uint32_t lo = opaque(q[u] & 0x0F0F0F0Fu);          // columns 8u + 0, 2, 4, 6
    const uint32_t hi = opaque((q[u] >> 4) & 0x0F0F0F0Fu);   // columns 8u + 1, 3, 5, 7
    a = __builtin_amdgcn_fdot2_f32_bf16(codes2_bf16<false>(lo), __builtin_bit_cast(bf16x2, xp[4 * u + 0]), a, false);
    a = __builtin_amdgcn_fdot2_f32_bf16(codes2_bf16<true>(lo), __builtin_bit_cast(bf16x2, xp[4 * u + 1]), a, false);
    b = __builtin_amdgcn_fdot2_f32_bf16(codes2_bf16<false>(hi), __builtin_bit_cast(bf16x2, xp[4 * u + 2]), b, false);
    b = __builtin_amdgcn_fdot2_f32_bf16(codes2_bf16<true>(hi), __builtin_bit_cast(bf16x2, xp[4 * u + 3]), b, false);
  }
  return a + b;
}

// Two code bytes as two float32 values q * 2^-9 (exact) in one conversion.
template <bool HI_WORD>
__device__ __forceinline__ f32x2 codes2_f32(uint32_t bytes) {
  return __builtin_amdgcn_cvt_pk_f32_fp8(bytes, HI_WORD);
}

// Eq. 3 from a scaled code: (q 2^-9) * (d 2^9) is the exact product d*q (both
// scalings are exact powers of two inside the value domain), so one FMA gives
// RN(d*q + m) -- the same bits as the plain definition.
__device__ __forceinline__ float eq3(float q_scaled, float d_times_512, float m) {
  return fmaf(q_scaled, d_times_512, m);
}

// Dequantizes 8 consecutive weights (one 32-bit word of codes) of a group to
// bf16 pairs in column order; d512 = d * 2^9 (see eq3).
__device__ __forceinline__ u32x4 dequant8_bf16(uint32_t codes, float d512, float m) {
  const uint32_t lo = opaque(codes & 0x0F0F0F0Fu);          // columns 0, 2, 4, 6
  const uint32_t hi = opaque((codes >> 4) & 0x0F0F0F0Fu);   // columns 1, 3, 5, 7
  const f32x2 a = codes2_f32<false>(lo), b = codes2_f32<true>(lo);
  const f32x2 e = codes2_f32<false>(hi), g = codes2_f32<true>(hi);
  u32x4 o;
  o[0] = pack_bf16x2(eq3(a[0], d512, m), eq3(e[0], d512, m));
  o[1] = pack_bf16x2(eq3(a[1], d512, m), eq3(e[1], d512, m));
  o[2] = pack_bf16x2(eq3(b[0], d512, m), eq3(g[0], d512, m));
  o[3] = pack_bf16x2(eq3(b[1], d512, m), eq3(g[1], d512, m));
  return o;
}

// ---- MXFP4 variant of the block --------------------------------------------
// Codes are FP4 E2M1 values and each group has one E8M0 scale byte e,
// X = 2^(e-127) (OCP MX v1.0).  gfx950 converts one code byte (low nibble =
// the even column) into two bf16 or float32 values times a float32 scale in
// one instruction; an FP4 value times a power of two in [2^-100, 2^100] is
// exact in both types.  Shifted into the float32 exponent field, e is X
// itself (e = 0, what a load past the end of a tile returns, gives +0).
__device__ __forceinline__ float e8m0_f32(uint32_t e) { return __uint_as_float(e << 23); }

__device__ __forceinline__ uint32_t load_u8(const uint8_t* p) { return (uint32_t)__builtin_nontemporal_load(p); }

template <int BYTE>
__device__ __forceinline__ uint32_t fp4x2_bf16(uint32_t codes, float scale) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(codes, scale, BYTE));
}

// 8 weights (one 32-bit word of codes) times X, as bf16 pairs in column order.
__device__ __forceinline__ u32x4 mx8_bf16(uint32_t codes, float X) {
  u32x4 o;
  o[0] = fp4x2_bf16<0>(codes, X);
  o[1] = fp4x2_bf16<1>(codes, X);
  o[2] = fp4x2_bf16<2>(codes, X);
  o[3] = fp4x2_bf16<3>(codes, X);
  return o;
}

// sum_i fp4(q_i) * x_i over one group (one 16-byte word of codes), x given as
// 16 bf16 pairs in natural column order.  The products are exact; v_dot2 adds
// two of them to the float32 accumulator.
__device__ __forceinline__ float group_dot_mx(u32x4 q, const uint32_t (&xp)[16]) {
  float a = 0.0f, b = 0.0f;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const uint32_t w = q[u];
    a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, fp4x2_bf16<0>(w, 1.0f)),
                                        __builtin_bit_cast(bf16x2, xp[4 * u + 0]), a, false);
    b = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, fp4x2_bf16<1>(w, 1.0f)),
                                        __builtin_bit_cast(bf16x2, xp[4 * u + 1]), b, false);
    a = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, fp4x2_bf16<2>(w, 1.0f)),
                                        __builtin_bit_cast(bf16x2, xp[4 * u + 2]), a, false);
    b = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, fp4x2_bf16<3>(w, 1.0f)),
                                        __builtin_bit_cast(bf16x2, xp[4 * u + 3]), b, false);
  }
  return a + b;
}

// Weight operand of the matrix kernels: a Q4NX blob, an MXFP4-variant blob or
// a plain bf16 matrix [N][K].
enum WFmt : int { kWBf16 = 0, kWQ4NX = 1, kWMX = 2 };
template <int F>
constexpr int wblock_bytes() {
  return F == kWMX ? kMxBlockBytes : kBlockBytes;
}

// ---------------------------------------------------------------------------
// q4nx_dequant / q4nx_mx_dequant: every weight, written row-major [N][K]
// ---------------------------------------------------------------------------
// One workgroup of 256 threads per block, 32 lanes per block row: lane j of a
// row handles columns 8j..8j+7 (one 32-bit word of codes, in group j/4), so a
// row's 32 lanes read 128 contiguous bytes of codes and write 512 (bf16) or
// 1024 (float32) contiguous bytes -- every store instruction writes whole
// lines.  Eight rows per pass, four passes per block.  (A lane per group, 64
// bytes of output per lane, writes a quarter of every line per instruction and
// ran at a fifth of this speed.)
template <int F>
__global__ __launch_bounds__(256) void dequant_kernel(const uint8_t* __restrict__ blob, int64_t N, int64_t K,
                                                      int64_t KB, int64_t nblocks, void* __restrict__ W,
                                                      int w_bf16) {
  constexpr int kBytes = wblock_bytes<F>();
  const int lr = threadIdx.x >> 5, j = threadIdx.x & 31;
  for (int64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
    const int64_t i = b / KB, jb = b - i * KB;
    const int64_t k = jb * kBlockCols + 8 * j;
    if (k >= K) continue;  // K is a multiple of 32: whole groups lie past K
    const uint8_t* blk = blob + b * kBytes;
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {
      const int r = 8 * pass + lr;
      const int64_t n = i * kBlockRows + r;
      if (n >= N) break;
      const uint32_t codes = *reinterpret_cast<const uint32_t*>(blk + 128 * r + 4 * j);
      const int gi = kGroupsPerRow * r + (j >> 2);
      u32x4 ob;
      float of[8];
      if constexpr (F == kWMX) {
        const float X = e8m0_f32(blk[kCodeBytes + gi]);
        if (w_bf16) {
          ob = mx8_bf16(codes, X);
        } else {
          const f32x2 a = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(codes, X, 0);
          const f32x2 c = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(codes, X, 1);
          const f32x2 e = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(codes, X, 2);
          const f32x2 g = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(codes, X, 3);
          of[0] = a[0]; of[1] = a[1]; of[2] = c[0]; of[3] = c[1];
          of[4] = e[0]; of[5] = e[1]; of[6] = g[0]; of[7] = g[1];
        }
      } else {
        const float d512 = bf16_to_f32(*reinterpret_cast<const uint16_t*>(blk + kCodeBytes + 2 * gi)) * 512.0f;
        const float m = bf16_to_f32(*reinterpret_cast<const uint16_t*>(blk + kCodeBytes + kScaleBytes + 2 * gi));
        if (w_bf16) {
          ob = dequant8_bf16(codes, d512, m);
        } else {
          const uint32_t lo = opaque(codes & 0x0F0F0F0Fu);          // columns 0, 2, 4, 6
          const uint32_t hi = opaque((codes >> 4) & 0x0F0F0F0Fu);   // columns 1, 3, 5, 7
          const f32x2 a = codes2_f32<false>(lo), c = codes2_f32<true>(lo);
          const f32x2 e = codes2_f32<false>(hi), g = codes2_f32<true>(hi);
          of[0] = eq3(a[0], d512, m); of[1] = eq3(e[0], d512, m);
          of[2] = eq3(a[1], d512, m); of[3] = eq3(e[1], d512, m);
          of[4] = eq3(c[0], d512, m); of[5] = eq3(g[0], d512, m);
          of[6] = eq3(c[1], d512, m); of[7] = eq3(g[1], d512, m);
        }
      }
      if (w_bf16) {
        *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(W) + n * K + k) = ob;
      } else {
        f32x4* out = reinterpret_cast<f32x4*>(static_cast<float*>(W) + n * K + k);
        out[0] = (f32x4){of[0], of[1], of[2], of[3]};
        out[1] = (f32x4){of[4], of[5], of[6], of[7]};
      }
    }
  }
}

// ---------------------------------------------------------------------------
// q4nx_quantize: float32 weights -> packed blob (the offline conversion)
// ---------------------------------------------------------------------------
// Per group of 32 consecutive input columns (Q4_1-style, Sec. 3.1.1):
//   w -> 0 if NaN, else clamped to [-2^100, 2^100] (keeps d and m in the
//   format's value domain); lo, hi = min, max (a zero minimum is +0);
//   d = RNE_bf16(RN(RN(hi - lo) / 15)), m = RNE_bf16(lo), magnitudes below
//   2^-100 flushed to a zero of the same sign;
//   q = the code whose Eq. 3 value is nearest to w (float64 differences),
//   the smaller code on a tie.
// The Eq. 3 levels L_q = fma(q, d, m) are non-decreasing in q, so the
// nearest level is found with two binary searches instead of a scan: c = the
// number of levels below w; the candidates are level c (the first >= w) and
// the first code whose level equals level c-1.
constexpr float kQuantClamp = 1.2676506002282294e30f;  // 2^100

__device__ __forceinline__ uint32_t bf16_rne_flushed(float v) {
  uint32_t b = pack_bf16x2(v, 0.0f) & 0xFFFFu;
  if ((b & 0x7FFFu) < (27u << 7)) b &= 0x8000u;  // |v| < 2^-100 -> signed zero
  return b;
}

// Number of codes q in 0..15 whose level fma(q, d, m) is below v.
__device__ __forceinline__ int levels_below(float v, float d, float m) {
  int c = 0;
#pragma unroll
  for (int s = 8; s >= 1; s >>= 1)
    if (fmaf((float)(c + s - 1), d, m) < v) c += s;
  if (c == 15 && fmaf(15.0f, d, m) < v) c = 16;
  return c;
}

__global__ __launch_bounds__(256) void quantize_kernel(const float* __restrict__ W, int64_t N, int64_t K, int64_t KB,
                                                       int64_t nblocks, uint8_t* __restrict__ blob) {
  const int t = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = 8 * t + (lane >> 3), c = lane & 7;
  for (int64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
    const int64_t i = b / KB, j = b - i * KB;
    const int64_t n = i * kBlockRows + r;
    const int64_t k0 = j * kBlockCols + kGroup * c;
    uint8_t* blk = blob + b * kBlockBytes;
    u32x4 codes = (u32x4){0u, 0u, 0u, 0u};
    uint32_t sb = 0, mb = 0;
    if (n < N && k0 < K) {
      float w[32];
      const f32x4* src = reinterpret_cast<const f32x4*>(W + n * K + k0);
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        const f32x4 x = src[v];
        w[4 * v + 0] = x[0];
        w[4 * v + 1] = x[1];
        w[4 * v + 2] = x[2];
        w[4 * v + 3] = x[3];
      }
      float lo = kQuantClamp, hi = -kQuantClamp;
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        const float x = w[e] != w[e] ? 0.0f : fminf(fmaxf(w[e], -kQuantClamp), kQuantClamp);
        w[e] = x;
        lo = fminf(lo, x);
        hi = fmaxf(hi, x);
      }
      lo = lo + 0.0f;  // a zero minimum is +0
      sb = bf16_rne_flushed((hi - lo) / 15.0f);
      mb = bf16_rne_flushed(lo);
      const float d = bf16_to_f32(sb), m = bf16_to_f32(mb);
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        const int cnt = levels_below(w[e], d, m);
        int q;
        if (cnt == 0) {
          q = 0;
        } else {
          const float l_lo = fmaf((float)(cnt - 1), d, m);
          // The first code with that level: cnt - 1 unless the level below is
          // the same value (a d small next to m), then the binary search.
          const int q_lo = (cnt == 1 || fmaf((float)(cnt - 2), d, m) < l_lo) ? cnt - 1 : levels_below(l_lo, d, m);
          if (cnt == 16) {
            q = q_lo;
          } else {
            const float l_hi = fmaf((float)cnt, d, m);
            const double dist_hi = (double)l_hi - (double)w[e];
            const double dist_lo = (double)w[e] - (double)l_lo;
            q = dist_hi < dist_lo ? cnt : q_lo;
          }
        }
        codes[e >> 3] |= (uint32_t)q << (4 * (e & 7));
      }
    }
    *reinterpret_cast<u32x4*>(blk + 1024 * t + 16 * lane) = codes;
    *reinterpret_cast<uint16_t*>(blk + kCodeBytes + 2 * (64 * t + lane)) = (uint16_t)sb;
    *reinterpret_cast<uint16_t*>(blk + kCodeBytes + kScaleBytes + 2 * (64 * t + lane)) = (uint16_t)mb;
  }
}

// q4nx_mx_quantize: float32 weights -> MXFP4-variant blob, with the lane
// mapping of quantize_kernel.  Per group (OCP MX v1.0 conversion): inputs
// taken into the domain as above; amax = max |w|; shared exponent
// e = floor(log2 amax) - 2 (2 = the largest FP4 exponent), clamped to
// [-100, 100], 0 for an all-zero group; each element w / 2^e rounded to the
// nearest FP4 magnitude -- the midpoints of {0, .5, 1, 1.5, 2, 3, 4, 6} go to
// the even mantissa -- saturating at 6, with the sign of w.  w / 2^e is exact
// (a power-of-two scaling; a result below 2^-126 only ever rounds to 0).
// The group maximum and the sign are read from the bit patterns, so that
// denormal inputs give the same exponent and sign whatever the denormal mode.
__device__ __forceinline__ uint32_t fp4_code(float w, float inv_x) {
  const float a = fabsf(w) * inv_x;
  const uint32_t m = (uint32_t)(a > 0.25f) + (uint32_t)(a >= 0.75f) + (uint32_t)(a > 1.25f) +
                     (uint32_t)(a >= 1.75f) + (uint32_t)(a > 2.5f) + (uint32_t)(a >= 3.5f) + (uint32_t)(a > 5.0f);
  const uint32_t bits = __float_as_uint(w);
  return m | ((bits >> 31) && (bits & 0x7FFFFFFFu) ? 8u : 0u);  // -0 keeps code 0
}

__global__ __launch_bounds__(256) void mx_quantize_kernel(const float* __restrict__ W, int64_t N, int64_t K,
                                                          int64_t KB, int64_t nblocks, uint8_t* __restrict__ blob) {
  const int t = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = 8 * t + (lane >> 3), c = lane & 7;
  for (int64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
    const int64_t i = b / KB, j = b - i * KB;
    const int64_t n = i * kBlockRows + r;
    const int64_t k0 = j * kBlockCols + kGroup * c;
    uint8_t* blk = blob + b * kMxBlockBytes;
    u32x4 codes = (u32x4){0u, 0u, 0u, 0u};
    uint32_t eb = kMxPadScale;  // padding: code 0 with scale 1
    if (n < N && k0 < K) {
      float w[32];
      const f32x4* src = reinterpret_cast<const f32x4*>(W + n * K + k0);
#pragma unroll
      for (int v = 0; v < 8; ++v) {
        const f32x4 x = src[v];
        w[4 * v + 0] = x[0];
        w[4 * v + 1] = x[1];
        w[4 * v + 2] = x[2];
        w[4 * v + 3] = x[3];
      }
      uint32_t amax = 0;  // bits of max |w|
#pragma unroll
      for (int e = 0; e < 32; ++e) {
        const float x = w[e] != w[e] ? 0.0f : (fabsf(w[e]) > kQuantClamp ? copysignf(kQuantClamp, w[e]) : w[e]);
        w[e] = x;
        amax = max(amax, __float_as_uint(x) & 0x7FFFFFFFu);
      }
      const int ex = amax == 0 ? 0 : max(-100, min(100, (int)(amax >> 23) - 127 - 2));
      eb = (uint32_t)(ex + 127);
      const float inv_x = __uint_as_float((uint32_t)(127 - ex) << 23);  // 2^-ex
#pragma unroll
      for (int e = 0; e < 32; ++e) codes[e >> 3] |= fp4_code(w[e], inv_x) << (4 * (e & 7));
    }
    *reinterpret_cast<u32x4*>(blk + 1024 * t + 16 * lane) = codes;
    blk[kCodeBytes + 64 * t + lane] = (uint8_t)eb;
  }
}

// ---------------------------------------------------------------------------
// q4nx_gemv / q4nx_gemv_batched: FusedDQP
// ---------------------------------------------------------------------------
// A workgroup owns a row group of R = 8*tq consecutive rows (tq = 4: a whole
// 32-row strip; 2: half a strip; 1: a quarter) and all of K.  Its W waves
// split the strip's blocks round-robin (block j goes to wave j % W); each
// wave accumulates, per lane, the rows 8t + l/8 (t = t0..t0+tq-1) of group
// l%8 as
//     acc += d_g * (sum_{k in g} q_k x_k) + m_g * S_g ,  S_g = sum_{k in g} x_k
// (Eq. 3 folded into Eq. 15), so the per-weight work is the exact code ->
// bf16 conversion and one v_dot2 per two weights.  A wave loads each block's
// x (512 bytes) together with the block's weights, in the same register slot,
// and stages it in its own LDS slot as bf16 pairs in the order the nibble
// split produces, forming the group sums with lane shuffles; groups are
// padded to 20 dwords so the eight groups a wave reads at once fall in
// distinct banks.  No wave waits for x beyond its own block, and there is no
// workgroup-wide staging phase or barrier before the first block.  At the end a 3-step
// butterfly adds the 8 groups of a row and the W waves' partial sums are added
// in wave order through LDS.  No workgroup talks to another, so there is no
// cross-XCD traffic and no device-wide fence.  The summation order is fixed
// for a given launch (results are reproducible call to call); it depends on
// the wave count W, which is chosen for the launch as a whole.
// Each wave prefetches its next block while computing the current one.
// For the MXFP4 variant the per-group term is X_g * (sum_{k in g} fp4(q_k) x_k)
// (no offset), with x staged in natural column order.
constexpr int kGemvMaxWaves = 16;
// A strip's weights are read 88 blocks at a time through one buffer
// descriptor (every Gemma3 K in one piece).
constexpr int kGemvChunkBlocks = 88;
constexpr int kGroupPadDw = 20;  // dwords per staged group (16 bf16 pairs + 4 pad: conflict-free reads)
constexpr int kRedFloats = kGemvMaxWaves * 32;
// Blocks in flight per wave (register slots), by row octets per wave.
constexpr int kGemvDepth4 = 1, kGemvDepth2 = 3, kGemvDepth1 = 4;
// Workgroups per CU of the streaming form (gemv_stream_kernel), LDS permitting.
constexpr int kGemvStreamPerCu = 4;

struct GemvJob {
  const uint8_t* blob;
  const uint16_t* x;
  void* y;
  int N, K, NS, KB;
  int tq;        // row octets per row group (1, 2 or 4)
  int nrg;       // row groups: NS * 4 / tq
  int waves;     // waves splitting K (depends on K only)
  int nwg;       // workgroups of this job (each loops over row groups)
  int wg_begin;  // first workgroup of this job in the launch
  int pad;
};

struct GemvArgs {
  GemvJob job[Q4NX_MAX_BATCH];
  int njobs;
  int y_bf16;
  int chunk_blocks;  // blocks per chunk: a strip's weights are read through one descriptor per chunk
  int pad;
};

// Registers of one in-flight block: TQ row octets of codes, scales, offsets
// (E8M0 scale bytes and no offsets for the MXFP4 variant).
template <int TQ>
struct GemvSlot {
  u32x4 q[TQ];
  uint32_t s[TQ], m[TQ];
  uint32_t xv[2];  // gemv_kernel: this lane's 4 bf16 of x for the block
};

// Buffer descriptor over one chunk of one strip (at most 88 blocks <= 440 KiB,
// so every offset fits the 32-bit descriptor range); raw, stride 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t chunk_rsrc(const uint8_t* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base), (short)0, bytes, 0x00020000);
}

// Cache policy of the weight loads: non-temporal (read once per call).
constexpr int kNtLoad = 2;

// Loads row octets t0..t0+TQ-1 of block `jj` of the chunk.  Every lane loads
// (all addresses lie inside the chunk); the caller skips blocks past the end
// with a wave-uniform branch.
template <int TQ, int F>
__device__ __forceinline__ void gemv_load(__amdgpu_buffer_rsrc_t rs, int jj, int t0, int lane, GemvSlot<TQ>& R) {
  const int boff = jj * wblock_bytes<F>();
#pragma unroll
  for (int t = 0; t < TQ; ++t) {
    const int tt = t0 + t;
    R.q[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, 16 * lane, boff + 1024 * tt, kNtLoad));
    if constexpr (F == kWMX) {
      R.s[t] = __builtin_amdgcn_raw_buffer_load_b8(rs, lane, boff + kCodeBytes + 64 * tt, kNtLoad);
    } else {
      R.s[t] = __builtin_amdgcn_raw_buffer_load_b16(rs, 2 * lane, boff + kCodeBytes + 128 * tt, kNtLoad);
      R.m[t] = __builtin_amdgcn_raw_buffer_load_b16(rs, 2 * lane, boff + kCodeBytes + kScaleBytes + 128 * tt, kNtLoad);
    }
  }
}

// x for one block, per wave: lane l = c + 8r (group c, r = 0..7) reads
// columns 32c + 4r .. 32c + 4r + 3 of the block (8 bytes; 512 contiguous
// bytes per wave), in the same ring slot as the block's weights.  The
// descriptor covers the chunk's columns inside K, so columns past K read 0.
__device__ __forceinline__ void gemv_load_x(__amdgpu_buffer_rsrc_t xr, int jj, int lane, uint32_t (&xv)[2]) {
  typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
  const u32x2 v = __builtin_bit_cast(
      u32x2, __builtin_amdgcn_raw_buffer_load_b64(xr, 2 * (kBlockCols * jj + 32 * (lane & 7) + 4 * (lane >> 3)), 0, 0));
  xv[0] = v[0];
  xv[1] = v[1];
}

// Stages one block's x in the wave's own LDS slot and returns the group sum
// S_g of this lane's group.  Q4NX: lane c + 8r writes the bf16 pairs of its 4
// columns, (x0,x2),(x1,x3) for even r, (x4,x6),(x5,x7) for odd r, so that each
// 8-column run u of a group holds (x0,x2),(x1,x3),(x4,x6),(x5,x7) at dwords
// 4u..4u+3 (slot of group c at dword c * kGroupPadDw).  S_g is formed in the
// same order as the workgroup-wide staging: per 8-column run
// ((x0+x1) + (x2+x3)) + (x4+x5) + (x6+x7), then (run0 + run1) + (run2 + run3).
// MXFP4 variant: the pairs in natural order, no sum.  The wave reads the slot
// right after writing it: a wave's LDS instructions are carried out in order,
// and the fence keeps the compiler from moving the reads above the writes.
template <int F>
__device__ __forceinline__ float gemv_stage_x(const uint32_t (&xv)[2], uint32_t* __restrict__ xw, int lane) {
  typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
  const int c = lane & 7, r = lane >> 3;
  uint32_t* dst = xw + c * kGroupPadDw + 2 * r;
  if constexpr (F == kWMX) {
    *reinterpret_cast<u32x2*>(dst) = (u32x2){xv[0], xv[1]};
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    return 0.0f;
  }
  const uint32_t pa = (xv[0] & 0xFFFFu) | (xv[1] << 16);           // (x0,x2) or (x4,x6)
  const uint32_t pb = (xv[0] >> 16) | (xv[1] & 0xFFFF0000u);       // (x1,x3) or (x5,x7)
  *reinterpret_cast<u32x2*>(dst) = (u32x2){pa, pb};
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  const float s01 = __uint_as_float(xv[0] << 16) + __uint_as_float(xv[0] & 0xFFFF0000u);
  const float s23 = __uint_as_float(xv[1] << 16) + __uint_as_float(xv[1] & 0xFFFF0000u);
  const float o01 = xor_lane<8>(s01), o23 = xor_lane<8>(s23);  // the odd lane's (x4+x5), (x6+x7)
  float sm = 0.0f;
  sm += s01;
  sm += s23;
  sm += o01;
  sm += o23;                       // the run's sum, on the even lanes
  sm += xor_lane<16>(sm);
  sm += xor_lane<32>(sm);
  const float se = xor_lane<8>(sm);
  return (r & 1) ? se : sm;
}

// One block's contribution to the lane's row sums: Eq. 15 with Eq. 3 folded
// in, x from the wave's slot (see gemv_stage_x).  Groups past K (block
// padding) contribute nothing whatever the padding holds.
template <int TQ, int F>
__device__ __forceinline__ void gemv_compute(const GemvSlot<TQ>& R, bool gvalid, const uint32_t* __restrict__ xg,
                                               float S, float (&acc)[4]) {
  uint32_t xp[16];
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const u32x4 xv = *reinterpret_cast<const u32x4*>(xg + 4 * v);
    if constexpr (F == kWMX) {
      xp[4 * v + 0] = xv[0];
      xp[4 * v + 1] = xv[1];
      xp[4 * v + 2] = xv[2];
      xp[4 * v + 3] = xv[3];
    } else {  // slot order (x0,x2),(x1,x3),(x4,x6),(x5,x7) -> the nibble split's order
      xp[4 * v + 0] = xv[0];
      xp[4 * v + 1] = xv[2];
      xp[4 * v + 2] = xv[1];
      xp[4 * v + 3] = xv[3];
    }
  }
  if constexpr (F == kWMX) {
#pragma unroll
    for (int t = 0; t < TQ; ++t) {
      const float dot = group_dot_mx(R.q[t], xp);
      acc[t] = fmaf(gvalid ? e8m0_f32(R.s[t]) : 0.0f, dot, acc[t]);
    }
    return;
  }
#pragma unroll
  for (int t = 0; t < TQ; ++t) {
    const float dot = group_dot_bf16(R.q[t], xp);
    const float d = gvalid ? bf16_to_f32(R.s[t]) : 0.0f;
    const float m = gvalid ? bf16_to_f32(R.m[t]) : 0.0f;
    acc[t] = fmaf(d, dot, acc[t]);
    acc[t] = fmaf(m, S, acc[t]);
  }
}

template <int TQ, int D, int F>
__global__ __launch_bounds__(64 * kGemvMaxWaves) void gemv_kernel(const GemvArgs args) {
  constexpr int kBytes = wblock_bytes<F>();
  // red: the waves' row sums; xw: each wave's x slot (one block of x).
  __shared__ float red[kRedFloats];
  __shared__ __attribute__((aligned(16))) uint32_t xw_all[kGemvMaxWaves][kGroupsPerRow * kGroupPadDw];

  const int wg = blockIdx.x;
  int jb = 0;
#pragma unroll
  for (int t = 1; t < Q4NX_MAX_BATCH; ++t)
    if (t < args.njobs && wg >= args.job[t].wg_begin) jb = t;
  const GemvJob& J = args.job[jb];

  // The wave index is uniform across a wave; saying so keeps every block
  // offset and branch derived from it in scalar registers.
  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c = lane & 7;
  const int W = J.waves;
  const bool wave_on = w < W;  // wave-uniform
  const int CB = args.chunk_blocks;
  const int nchunks = (J.KB + CB - 1) / CB;
  uint32_t* const xw = xw_all[wave_on ? w : 0];

  for (int rg = wg - J.wg_begin; rg < J.nrg; rg += J.nwg) {
    const int row0 = rg * 8 * TQ;
    const int strip = row0 >> 5, t0 = (row0 & 31) >> 3;
    const uint8_t* sblob = J.blob + (size_t)strip * J.KB * kBytes;
    float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};

    for (int ch = 0; ch < nchunks; ++ch) {
      const int jc0 = ch * CB;
      const int nb = min(CB, J.KB - jc0);
      const __amdgpu_buffer_rsrc_t rs = chunk_rsrc(sblob + (size_t)jc0 * kBytes, nb * kBytes);
      const int kvalid = J.K - jc0 * kBlockCols;  // columns of this chunk inside K
      const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint16_t*>(J.x + (size_t)jc0 * kBlockCols), (short)0, 2 * min(kvalid, nb * kBlockCols),
          0x00020000);
      if (!wave_on) continue;
      // Ring of D register slots: block w + iW lives in slot i % D and the
      // slot is refilled with block w + (i + D)W right after it is consumed;
      // each slot carries the block's x with its weights, so a wave starts
      // on its first block as soon as that block has arrived.
      GemvSlot<TQ> buf[D];
#pragma unroll
      for (int d = 0; d < D; ++d)
        if (w + d * W < nb) {
          gemv_load_x(xr, w + d * W, lane, buf[d].xv);
          gemv_load<TQ, F>(rs, w + d * W, t0, lane, buf[d]);
        }
      for (int i0 = 0; w + i0 * W < nb; i0 += D) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
          const int jj = w + (i0 + d) * W;
          if (jj < nb) {
            const float S = gemv_stage_x<F>(buf[d].xv, xw, lane);
            gemv_compute<TQ, F>(buf[d], jj * kBlockCols + kGroup * c < kvalid, xw + c * kGroupPadDw, S, acc);
            if (jj + D * W < nb) {
              gemv_load_x(xr, jj + D * W, lane, buf[d].xv);
              gemv_load<TQ, F>(rs, jj + D * W, t0, lane, buf[d]);
            }
          }
        }
      }
    }

    // Add the 8 groups of each row: lanes 8r'..8r'+7 hold row octet t, row r'.
#pragma unroll
    for (int t = 0; t < TQ; ++t) {
      acc[t] += xor_lane<1>(acc[t]);
      acc[t] += xor_lane<2>(acc[t]);
      acc[t] += xor_lane<4>(acc[t]);
    }
    // Lane with c == t (t < TQ) holds row 8t + l/8 of the row group.
    if (wave_on && c < TQ) {
      const float v = (c == 0) ? acc[0] : (c == 1) ? acc[1] : (c == 2) ? acc[2] : acc[3];
      red[w * 32 + 8 * c + (lane >> 3)] = v;
    }
    __syncthreads();
    if (threadIdx.x < 8 * TQ) {
      float sum = 0.0f;
      for (int q = 0; q < W; ++q) sum += red[q * 32 + threadIdx.x];
      const int64_t n = (int64_t)row0 + threadIdx.x;
      if (n < J.N) {
        if (args.y_bf16)
          static_cast<uint16_t*>(J.y)[n] = f32_to_bf16_bits(sum);
        else
          static_cast<float*>(J.y)[n] = sum;
      }
    }
    __syncthreads();  // red[] is rewritten by the next row group
  }
}

// Persistent streaming form of gemv_kernel, for launches whose K fits one
// chunk (every Gemma3 K).  A job's row groups are dealt to a bounded number
// of workgroups, rg = r0, r0 + nwg, ...; each wave streams its blocks of all
// its row groups (w, w + W, ... of each), each block with its x, through one
// ring of D register slots that runs on across row groups, so the next row
// group's loads are in flight while the current one's rows are added up and
// stored.  The arithmetic and the order of every sum are those of
// gemv_kernel (same waves per row group), hence the same bits.  Every wave
// meets the same barriers: two per row group.
template <int TQ, int D, int F>
__global__ __launch_bounds__(64 * kGemvMaxWaves) void gemv_stream_kernel(const GemvArgs args) {
  constexpr int kBytes = wblock_bytes<F>();
  __shared__ float red[kRedFloats];
  __shared__ __attribute__((aligned(16))) uint32_t xw_all[kGemvMaxWaves][kGroupsPerRow * kGroupPadDw];

  const int wg = blockIdx.x;
  int jb = 0;
#pragma unroll
  for (int t = 1; t < Q4NX_MAX_BATCH; ++t)
    if (t < args.njobs && wg >= args.job[t].wg_begin) jb = t;
  const GemvJob& J = args.job[jb];

  const int lane = threadIdx.x & 63, w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c = lane & 7;
  const int W = J.waves, nb = J.KB;
  const bool wave_on = w < W;  // wave-uniform
  const int r0 = wg - J.wg_begin;
  const int nrg = r0 < J.nrg ? (J.nrg - 1 - r0) / J.nwg + 1 : 0;  // row groups of this workgroup
  if (nrg == 0) return;                                           // the whole workgroup
  const int nbw = wave_on ? (nb - w + W - 1) / W : 0;              // this wave's blocks per row group
  const int Q = nbw * nrg;
  const int kvalid = J.K;
  const int sbytes = nb * kBytes;  // bytes of one strip
  uint32_t* const xw = xw_all[wave_on ? w : 0];
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(J.x), (short)0, 2 * J.K, 0x00020000);

  // Load cursor: row group lk of this workgroup, this wave's block ljq of it.
  int lk = 0, ljq = 0;
  auto load_next = [&](GemvSlot<TQ>& R, int& jj) {
    const int row0 = (r0 + lk * J.nwg) * 8 * TQ;
    jj = w + ljq * W;
    gemv_load_x(xr, jj, lane, R.xv);
    gemv_load<TQ, F>(chunk_rsrc(J.blob + (size_t)(row0 >> 5) * sbytes, sbytes), jj, (row0 & 31) >> 3, lane, R);
    if (++ljq == nbw) {
      ljq = 0;
      ++lk;
    }
  };

  GemvSlot<TQ> buf[D];
  int jjs[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    jjs[d] = 0;
    if (d < Q) load_next(buf[d], jjs[d]);
  }

  // Row group k of this workgroup is complete in every wave: add the 8 groups
  // of each row, then the W waves' sums in wave order, and store.
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  auto finish = [&](int k) {
#pragma unroll
    for (int t = 0; t < TQ; ++t) {
      acc[t] += xor_lane<1>(acc[t]);
      acc[t] += xor_lane<2>(acc[t]);
      acc[t] += xor_lane<4>(acc[t]);
    }
    if (wave_on && c < TQ) {
      const float v = (c == 0) ? acc[0] : (c == 1) ? acc[1] : (c == 2) ? acc[2] : acc[3];
      red[w * 32 + 8 * c + (lane >> 3)] = v;
    }
    __syncthreads();
    if (threadIdx.x < 8 * TQ) {
      float sum = 0.0f;
      for (int q = 0; q < W; ++q) sum += red[q * 32 + threadIdx.x];
      const int64_t n = (int64_t)(r0 + k * J.nwg) * 8 * TQ + threadIdx.x;
      if (n < J.N) {
        if (args.y_bf16)
          static_cast<uint16_t*>(J.y)[n] = f32_to_bf16_bits(sum);
        else
          static_cast<float*>(J.y)[n] = sum;
      }
    }
    __syncthreads();  // red[] is rewritten for the next row group
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = 0.0f;
  };

  if (Q == 0) {  // a wave without blocks still meets every barrier
    for (int k = 0; k < nrg; ++k) finish(k);
    return;
  }
  // Ring of D slots: block q of the wave's stream lives in slot q % D and the
  // slot is refilled with block q + D right after it is consumed.
  int ck = 0, cjq = 0;
  for (int q0 = 0; q0 < Q; q0 += D) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int q = q0 + d;
      if (q < Q) {
        const int jj = jjs[d];
        const float S = gemv_stage_x<F>(buf[d].xv, xw, lane);
        gemv_compute<TQ, F>(buf[d], jj * kBlockCols + kGroup * c < kvalid, xw + c * kGroupPadDw, S, acc);
        if (q + D < Q) load_next(buf[d], jjs[d]);
        if (++cjq == nbw) {
          finish(ck);
          cjq = 0;
          ++ck;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// q4nx_gemm: fused dequant + bf16 MFMA matrix product
// ---------------------------------------------------------------------------
// Every kernel below walks K in steps of 64 (two quantization groups) and
// feeds v_mfma_f32_32x32x16_bf16 from LDS: the X tile as loaded (bf16) and
// the W tile dequantized with Eq. 3 in float32 and rounded to bf16 (the
// paper's prefill dequantizes to bf16 before the MM).  LDS rows are padded to
// 72 elements (144 B) so that the 16-byte fragment reads of 8 consecutive
// rows, and the 16-byte tile writes, hit distinct banks.  Each output is the
// float32 sum of its MFMA chain over K in increasing order, so every kernel
// and every tile shape gives the same bits.  MXFP4-variant weights take the
// same path with the Eq. 3 step replaced by the exact FP4 x scale conversion.
constexpr int kBK = 64;
constexpr int kLdsStride = kBK + 8;  // bf16 elements per LDS row

// Tile order.  Workgroups are dispatched round-robin over the 8 XCDs, each
// with its own L2.  Workgroup w runs on XCD w % 8, so XCD x is given the
// contiguous range of logical tiles [x*T/8, (x+1)*T/8); logical tiles are
// ordered in groups of kGroupM tile rows, column by column, so the tiles an
// XCD runs at the same time share a few X row blocks and W column blocks in
// its L2 instead of streaming the whole operands from the memory-side cache.
constexpr int kXcds = 8;
constexpr int kGroupM = 4;

__device__ __forceinline__ void gemm_tile_of(int wg, int ntiles, int tiles_n, int& bm, int& bn) {
  const int x = wg % kXcds, l = wg / kXcds;
  const int base = ntiles / kXcds, rem = ntiles % kXcds;
  const int t = x * base + min(x, rem) + l;
  const int tiles_m = ntiles / tiles_n;
  const int group = t / (kGroupM * tiles_n);
  const int rows = min(kGroupM, tiles_m - group * kGroupM);  // tile rows in this (last) group
  const int r = t - group * kGroupM * tiles_n;
  bm = group * kGroupM + r % rows;
  bn = r / rows;
}


// Output of one wave's TI x TJ accumulator blocks when its whole 32TI x 32TJ
// sub-tile lies inside the matrix.  base (uniform over the wave) is the
// sub-tile's first element, ldy
// the row stride in elements (float32, or bf16 when bf16 != 0).  In the MFMA
// layout, element e of lane l is column l%32 and row 8(e/4) + 4(l/32) + e%4
// of its block: only the lane's own part of an address varies across the
// wave, so every element is one buffer store whose block and row offset is a
// scalar -- no per-element 64-bit address arithmetic and no bounds tests,
// which made the plain per-element stores several times longer than the
// memory needs to take them.
// Offsets inside a wave's sub-tile are 32-bit: its extent is below 2^31 bytes
// for every row stride below 2^21 elements (at most 256 rows of 4 bytes).
// Wider rows take the checked per-element stores, which address in 64 bits.
constexpr int kFastStoreMaxLdy = 1 << 21;

template <int TI, int TJ>
__device__ __forceinline__ void store_wave_tile(const f32x16 (&acc)[TI][TJ], void* base, int ldy, int bf16) {
  // The lane index is recomputed here rather than kept live across the K loop.
  const int lane = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
  const unsigned esz = bf16 ? 2u : 4u, rb = (unsigned)ldy * esz;
  // base is the same in every lane; saying so keeps the descriptor scalar
  // (otherwise each store may become a loop over distinct descriptors).
  const uint64_t bp = reinterpret_cast<uint64_t>(base);
  // (readfirstlane yields an int: each half goes through uint32_t so that the
  // low word is not sign-extended into the high one.)
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(bp >> 32));
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)bp);
  void* const ub = reinterpret_cast<void*>(((uint64_t)hi << 32) | (uint64_t)lo);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      ub, (short)0, (int)((32 * TI - 1) * rb + 32 * TJ * esz), 0x00020000);
  const int vo = (int)(4u * (unsigned)(lane >> 5) * rb + (unsigned)(lane & 31) * esz);
  if (bf16) {
#pragma unroll
    for (int a = 0; a < TI; ++a)
#pragma unroll
      for (int b = 0; b < TJ; ++b)
#pragma unroll
        for (int e = 0; e < 16; e += 2) {  // rows r and r + 1
          const uint32_t v = pack_bf16x2(acc[a][b][e], acc[a][b][e + 1]);
          const int so = (int)((unsigned)(32 * a + 8 * (e >> 2) + (e & 3)) * rb + 64u * b);
          __builtin_amdgcn_raw_buffer_store_b16((unsigned short)v, rs, vo, so, 0);
          __builtin_amdgcn_raw_buffer_store_b16((unsigned short)(v >> 16), rs, vo, so + (int)rb, 0);
        }
  } else {
#pragma unroll
    for (int a = 0; a < TI; ++a)
#pragma unroll
      for (int b = 0; b < TJ; ++b)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int so = (int)((unsigned)(32 * a + 8 * (e >> 2) + (e & 3)) * rb + 128u * b);
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(acc[a][b][e]), rs, vo, so, 0);
        }
  }
}

// ---- 256 x 256 tile, one wave per SIMD ------------------------------------
// Four waves in a 2 x 2 grid, each owning a 128 x 128 sub-tile: 16 MFMA
// accumulators (256 accumulation registers, which live in the AGPR half of the
// register file), so each 16-deep K slice costs 16 MFMAs against 8 fragment
// reads -- half the LDS read traffic per MFMA of a 128 x 64 wave tile.  With
// a single wave per SIMD nothing hides a stall, so the instruction order is
// fixed by hand: a K step is four blocks of 16 MFMA slots, each slot one MFMA
// plus a fixed share of the other work, fenced so the compiler keeps it there:
//   slots  0-15  MFMAs of K slice 0 | fragment reads of slice 1 | part of
//                the next step's tiles written to the other LDS stage (X, or
//                bf16 W) | weight group 0 of the next step dequantized (a
//                quarter of 8 columns per slot)
//   slots 16-31  slice 1 | reads of slice 2 | more of the tiles | weight
//                group 1 dequantized
//   slots 32-47  slice 2 | reads of slice 3 | the rest of a bf16 W tile
//   barrier      (the other stage is complete; this stage's reads are done)
//   slots 48-63  slice 3 | reads of slice 0 of the next step
// with the global loads of step + 3 issued as their registers free up (the
// exact placement is given at the step function below).  The raw operands of
// a step are loaded into registers two steps ahead.  X and
// W are read through buffer descriptors limited to the tile's rows and strips;
// in the last step of a K that is not a multiple of 64 the columns past K are
// given an offset past the descriptor's end, which reads as zero -- code 0,
// scale 0 and offset 0 give w = +0 (code 0 with E8M0 byte 0 as well) -- so no
// mask is needed anywhere else.  X
// rows past M and W strips past the matrix are clamped to the last valid one;
// their outputs are never stored.
constexpr int kWideThreads = 256;
constexpr int kMaxSplit = 4;  // K segments of a split-K launch, at most
constexpr int kWideLdsBytes = 2 * 2 * 256 * kLdsStride * 2;  // two stages of X and W
constexpr int64_t kWideMaxK = int64_t(1) << 22;               // 256 rows x K x 2 B < 2^31

// Raw operands of one K step held by one thread.  X (and bf16 W): rows
// tid/8 + 32i, columns 8(tid%8)..+7 of the step.  Packed W: codes, scale and
// offset (no offset for the MXFP4 variant) of group (row tid/2 + 128g, half
// tid%2 of the step).
template <int WF>
struct WideRegs {
  u32x4 x[8];
  u32x4 q[2];
  uint32_t s[2], m[2];
};
template <>
struct WideRegs<kWBf16> {
  u32x4 x[8];
  u32x4 w[8];
};

// Dequantization of one packed weight group (16 code bytes, its scale s and
// offset m as loaded) in 16 pieces: piece p handles a quarter of the 8
// columns 8(p/4)..+7 (Eq. 3, as in dequant8_bf16; for the MXFP4 variant one
// FP4 x scale conversion of a code byte, as in mx8_bf16), and the last
// quarter stores the 8 bf16 weights at dst + 8(p/4).  The hand-scheduled
// GEMM kernels spread the pieces over their MFMA slots, one per slot.
template <int WF>
struct GroupDequant {
  uint32_t lo = 0, hi = 0;
  float d = 0.0f, m = 0.0f;
  f32x2 a, e, b, g;
  u32x4 o;
  __device__ __forceinline__ void piece(const u32x4& q, uint32_t s, uint32_t mo, int p, uint16_t* dst) {
    const int u = p >> 2, qt = p & 3;
    if constexpr (WF == kWMX) {
      if (p == 0) d = e8m0_f32(s);
      const uint32_t w = q[u];
      if (qt == 0) o[0] = fp4x2_bf16<0>(w, d);
      else if (qt == 1) o[1] = fp4x2_bf16<1>(w, d);
      else if (qt == 2) o[2] = fp4x2_bf16<2>(w, d);
      else {
        o[3] = fp4x2_bf16<3>(w, d);
        *reinterpret_cast<u32x4*>(dst + 8 * u) = o;
      }
    } else {
      if (qt == 0) {
        if (u == 0) {
          d = bf16_to_f32(s) * 512.0f;
          m = bf16_to_f32(mo);
        }
        lo = opaque(q[u] & 0x0F0F0F0Fu);
        hi = opaque((q[u] >> 4) & 0x0F0F0F0Fu);
        a = codes2_f32<false>(lo);
      } else if (qt == 1) {
        e = codes2_f32<false>(hi);
        o[0] = pack_bf16x2(eq3(a[0], d, m), eq3(e[0], d, m));
        o[1] = pack_bf16x2(eq3(a[1], d, m), eq3(e[1], d, m));
      } else if (qt == 2) {
        b = codes2_f32<true>(lo);
        g = codes2_f32<true>(hi);
        o[2] = pack_bf16x2(eq3(b[0], d, m), eq3(g[0], d, m));
      } else {
        o[3] = pack_bf16x2(eq3(b[1], d, m), eq3(g[1], d, m));
        *reinterpret_cast<u32x4*>(dst + 8 * u) = o;
      }
    }
  }
};

// WF: W is a packed Q4NX or MXFP4-variant matrix (dequantized on the fly), or
// bf16 [N][K], whose tile is staged exactly like the X tile.
// Split K: workgroup (x, y) computes tile x over K steps [y*ksteps,
// min((y+1)*ksteps, all steps)) and, when `part` is given, writes its float32
// partial product to part + y*M*ldy (row stride ldy) instead of Y.
template <bool KTAIL, int WF>
__global__ __launch_bounds__(kWideThreads) void gemm256_kernel(const uint16_t* __restrict__ X,
                                                               const uint8_t* __restrict__ wsrc,
                                                               void* __restrict__ Y, int M, int N, int K, int ldy,
                                                               int KB, int NS, int tiles_n, int y_bf16, int ksteps,
                                                               float* __restrict__ part) {
  constexpr int TI = 4, TJ = 4;
  extern __shared__ __attribute__((aligned(16))) uint16_t gl[];
  uint16_t* const xs0 = gl;                          // [2][256][72]
  uint16_t* const ws0 = gl + 2 * 256 * kLdsStride;   // [2][256][72]

  int bm, bn;
  gemm_tile_of(blockIdx.x, gridDim.x, tiles_n, bm, bn);
  const int m0 = bm * 256, n0 = bn * 256;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  const int rows_x = min(256, M - m0);
  const __amdgpu_buffer_rsrc_t rsx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(X + (size_t)m0 * K), (short)0, rows_x * K * 2, 0x00020000);
  constexpr bool WQ4 = WF != kWBf16;  // packed weights
  constexpr int kBB = wblock_bytes<WF>();
  const int s0 = n0 >> 5, nst = min(8, NS - s0), rows_w = min(256, N - n0);
  const __amdgpu_buffer_rsrc_t rsw =
      WQ4 ? __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(wsrc + (size_t)s0 * KB * kBB), (short)0,
                                              nst * KB * kBB, 0x00020000)
          : __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(wsrc + (size_t)n0 * K * 2), (short)0,
                                              rows_w * K * 2, 0x00020000);
  constexpr int kPastEnd = 0x7FFFFFF0;  // beyond every descriptor: loads return 0
  // Global loads per thread and K step.
  constexpr int kLoads = WF == kWQ4NX ? 14 : WF == kWMX ? 12 : 16;

  const int c8 = tid & 7, half = tid & 1;
  int vx[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) vx[i] = (min((tid >> 3) + 32 * i, rows_x - 1) * K + 8 * c8) * 2;
  int vq[2], vs[2], vw[8];
  if constexpr (WQ4) {
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const int r = (tid >> 1) + 128 * g;
      const int st = min(r >> 5, nst - 1), rr = r & 31;
      vq[g] = st * KB * kBB + 128 * rr + 16 * half;
      vs[g] = st * KB * kBB + kCodeBytes + (WF == kWMX ? 1 : 2) * (8 * rr + half);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) vw[i] = (min((tid >> 3) + 32 * i, rows_w - 1) * K + 8 * c8) * 2;
  }
  // K steps of this workgroup's segment: sb .. sb + nsteps - 1.
  const int sb = blockIdx.y * ksteps;
  const int nsteps = min((K + kBK - 1) / kBK, sb + ksteps) - sb;

  f32x16 acc[TI][TJ];
#pragma unroll
  for (int a = 0; a < TI; ++a)
#pragma unroll
    for (int b = 0; b < TJ; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.0f;

  // Global loads of step t of the segment (clamped to its last step) into R,
  // one of the kLoads loads per call, so that they can be spread over MFMA
  // slots.
  auto load1 = [&](WideRegs<WF>& R, int t, int i) {
    const int k0 = (sb + min(t, nsteps - 1)) * kBK;
    const int sq = (k0 >> 8) * kBB + 16 * ((k0 & 255) >> 5);
    const int ss = (k0 >> 8) * kBB + (WF == kWMX ? 1 : 2) * ((k0 & 255) >> 5);
    const bool okx = !KTAIL || k0 + 8 * c8 < K;
    const bool okw = !KTAIL || k0 + kGroup * half < K;
    if (i < 8) {
      if (!KTAIL)
        R.x[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsx, vx[i], 2 * k0, 0));
      else
        R.x[i] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsx, okx ? vx[i] + 2 * k0 : kPastEnd, 0, 0));
      return;
    }
    if constexpr (!WQ4) {
      if (!KTAIL)
        R.w[i - 8] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsw, vw[i - 8], 2 * k0, 0));
      else
        R.w[i - 8] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsw, okx ? vw[i - 8] + 2 * k0 : kPastEnd, 0, 0));
    } else if (i < 10) {
      const int g = i - 8;
      R.q[g] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsw, okw ? vq[g] + sq : kPastEnd, 0, kNtLoad));
    } else if (i < 12) {
      const int g = i - 10;
      if constexpr (WF == kWMX)
        R.s[g] = __builtin_amdgcn_raw_buffer_load_b8(rsw, okw ? vs[g] + ss : kPastEnd, 0, kNtLoad);
      else
        R.s[g] = __builtin_amdgcn_raw_buffer_load_b16(rsw, okw ? vs[g] + ss : kPastEnd, 0, kNtLoad);
    } else {
      const int g = i - 12;
      R.m[g] = __builtin_amdgcn_raw_buffer_load_b16(rsw, okw ? vs[g] + ss + kScaleBytes : kPastEnd, 0, kNtLoad);
    }
  };
  auto xs_row = [&](int st) { return xs0 + st * 256 * kLdsStride + (tid >> 3) * kLdsStride + 8 * c8; };
  auto ws_row = [&](int st, int g) {
    return ws0 + st * 256 * kLdsStride + ((tid >> 1) + 128 * g) * kLdsStride + kGroup * half;
  };
  // Fragment i of K slice kq, in first-use order A0, B0, B1, B2, B3, A1, A2, A3.
  const int fa = (128 * wm + (lane & 31)) * kLdsStride + 8 * (lane >> 5);
  const int fb = (128 * wn + (lane & 31)) * kLdsStride + 8 * (lane >> 5);
  auto read1 = [&](int st, int kq, bf16x8 (&A)[TI], bf16x8 (&B)[TJ], int i) {
    const uint16_t* xs = xs0 + st * 256 * kLdsStride + fa + 16 * kq;
    const uint16_t* ws = ws0 + st * 256 * kLdsStride + fb + 16 * kq;
    if (i == 0) A[0] = *reinterpret_cast<const bf16x8*>(xs);
    else if (i <= 4) B[i - 1] = *reinterpret_cast<const bf16x8*>(ws + 32 * (i - 1) * kLdsStride);
    else A[i - 4] = *reinterpret_cast<const bf16x8*>(xs + 32 * (i - 4) * kLdsStride);
  };
  auto mma1 = [&](const bf16x8 (&A)[TI], const bf16x8 (&B)[TJ], int i) {
    acc[i >> 2][i & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[i >> 2], B[i & 3], acc[i >> 2][i & 3], 0, 0, 0);
  };
  // Weight group g of the next step dequantized piece by piece.
  GroupDequant<WF> gdq;
  auto wpiece = [&](const WideRegs<WF>& R, int st, int g, int p) {
    if constexpr (WQ4) gdq.piece(R.q[g], R.s[g], WF == kWMX ? 0u : R.m[g], p, ws_row(st, g));
  };
  // bf16 W: chunk i of the thread's W rows, staged like X.
  auto wchunk = [&](const WideRegs<WF>& R, int st, int i) {
    if constexpr (!WQ4)
      *reinterpret_cast<u32x4*>(xs_row(st) + 2 * 256 * kLdsStride + 32 * i * kLdsStride) = R.w[i];
  };

  // One K step: MFMAs of step s from stage s&1 while step s+1 (held in Rs) is
  // written to the other stage and step s+3 is loaded into Rs.
  //
  // Placement of the LDS accesses.  A slot is one MFMA, 32 clocks, in which
  // the CU's LDS serves about six 1 KiB wave reads or two and a half wave
  // writes (measured on MI355X: ~190 and ~78 bytes per clock), and every
  // slice reads its 8 fragments of the next slice.  The writes of the
  // other stage must land before the barrier, so they are spread over the
  // slices before it instead of being packed into one:
  //   bf16 W (16 writes: x0..x7, w0..w7), odd slots from 1: slice 0 x0..x5,
  //     slice 1 x6 x7 w0..w3, slice 2 w4..w7 -- at most 14 accesses in a
  //     slice; fragment reads on the even slots (slice 2: slots 0, 2, 4, 6,
  //     8-11, well before the barrier);
  //   packed W: reads on the even slots of slices 0-1, X at slots 1, 5, 9, 13
  //     (x0..x3 in slice 0, x4..x7 in slice 1) between the dequantized W
  //     writes at slots 3, 7, 11, 15.  (With a K tail the X writes stay at
  //     slots 8-15 of slice 0: the interleaved form costs that instantiation
  //     a register spill.)
  // The order of the MFMAs, hence every result bit, does not depend on this.
  constexpr bool kSpreadPacked = WQ4 && !KTAIL;
  auto stage_write = [&](WideRegs<WF>& Rs, uint16_t* xsn, int nxt, int slice, int i) {
    if (!(i & 1)) return;
    const int o = i >> 1;
    if constexpr (!WQ4) {
      if (slice < 2 ? o >= 6 : o >= 4) return;
      const int k = slice * 6 + o;
      if (k < 8)
        *reinterpret_cast<u32x4*>(xsn + 32 * k * kLdsStride) = Rs.x[k];
      else
        wchunk(Rs, nxt, k - 8);
    } else if constexpr (kSpreadPacked) {
      if (slice < 2 && (o & 1) == 0) {
        const int k = 4 * slice + (o >> 1);
        *reinterpret_cast<u32x4*>(xsn + 32 * k * kLdsStride) = Rs.x[k];
      }
    }
  };
  const auto read_slot = [](int slice, int i) {
    if (!WQ4 || kSpreadPacked) {
      if (slice < 2) return (i & 1) ? -1 : i >> 1;
      if (!WQ4) return i < 8 ? ((i & 1) ? -1 : i >> 1) : (i < 12 ? i - 4 : -1);
    }
    return i < 8 ? i : -1;
  };
  // Global loads of step s + 3 go out as soon as their registers are free:
  // one slot after the write that empties them (bf16 W, and X of packed W),
  // and a packed W group in the slice after the one that dequantizes it.  So
  // they spread over slices 0-2 instead of forming one burst in slice 2, and
  // leave up to two slices earlier.  (With a K tail, packed W keeps the
  // original order: all loads in slice 2, load i at slot i.)
  auto early_load = [&](WideRegs<WF>& Rs, int s, int slice, int i) {
    if constexpr (!WQ4) {
      // load k one slot after write k (odd slot 2o+1 of its slice; the
      // per-slice write counts of stage_write)
      if ((i & 1) || i == 0) return;
      constexpr int c[3] = {6, 6, 4};
      const int o = (i >> 1) - 1;
      if (o >= c[slice]) return;
      const int k = (slice > 0 ? c[0] : 0) + (slice > 1 ? c[1] : 0) + o;
      load1(Rs, s + 3, k);
    } else if constexpr (kSpreadPacked) {
      if (slice < 2 && (i & 3) == 2) load1(Rs, s + 3, 4 * slice + (i >> 2));  // x after its write at i - 1
      // W group 0 after slice 0's dequant, group 1 after slice 1's
      if (slice == 1 && (i & 1) && i < 7) {
        const int j = i >> 1;  // 0 q, 1 s, 2 m
        const int idx = 8 + 2 * j;
        if (idx < kLoads) load1(Rs, s + 3, idx);
      }
      if (slice == 2 && !(i & 1) && i < 6) {
        const int j = i >> 1;
        const int idx = 9 + 2 * j;
        if (idx < kLoads) load1(Rs, s + 3, idx);
      }
    }
  };
  bf16x8 A0[TI], B0[TJ], A1[TI], B1[TJ];
  auto step = [&](int s, WideRegs<WF>& Rs) {
    const int cur = s & 1, nxt = cur ^ 1;
    uint16_t* xsn = xs_row(nxt);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      mma1(A0, B0, i);
      if (read_slot(0, i) >= 0) read1(cur, 1, A1, B1, read_slot(0, i));
      if constexpr (WQ4 && !kSpreadPacked) {
        if (i >= 8) *reinterpret_cast<u32x4*>(xsn + 32 * (i - 8) * kLdsStride) = Rs.x[i - 8];
      } else {
        stage_write(Rs, xsn, nxt, 0, i);
      }
      wpiece(Rs, nxt, 0, i);
      early_load(Rs, s, 0, i);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      mma1(A1, B1, i);
      if (read_slot(1, i) >= 0) read1(cur, 2, A0, B0, read_slot(1, i));
      stage_write(Rs, xsn, nxt, 1, i);
      wpiece(Rs, nxt, 1, i);
      early_load(Rs, s, 1, i);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      mma1(A0, B0, i);
      if (read_slot(2, i) >= 0) read1(cur, 3, A1, B1, read_slot(2, i));
      stage_write(Rs, xsn, nxt, 2, i);
      if constexpr (WQ4 && !kSpreadPacked) {
        if (i < kLoads) load1(Rs, s + 3, i);
      } else {
        early_load(Rs, s, 2, i);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      mma1(A1, B1, i);
      if (i < 8) read1(nxt, 0, A0, B0, i);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  WideRegs<WF> R0, R1;
#pragma unroll
  for (int i = 0; i < kLoads; ++i) load1(R0, 0, i);
#pragma unroll
  for (int i = 0; i < kLoads; ++i) load1(R1, 1, i);
  {
    uint16_t* xs = xs_row(0);
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<u32x4*>(xs + 32 * i * kLdsStride) = R0.x[i];
    if constexpr (WF == kWMX) {
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const float X = e8m0_f32(R0.s[g]);
#pragma unroll
        for (int u = 0; u < 4; ++u) *reinterpret_cast<u32x4*>(ws_row(0, g) + 8 * u) = mx8_bf16(R0.q[g][u], X);
      }
    } else if constexpr (WQ4) {
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const float d512 = bf16_to_f32(R0.s[g]) * 512.0f, m = bf16_to_f32(R0.m[g]);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          *reinterpret_cast<u32x4*>(ws_row(0, g) + 8 * u) = dequant8_bf16(R0.q[g][u], d512, m);
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) wchunk(R0, 0, i);
    }
  }
#pragma unroll
  for (int i = 0; i < kLoads; ++i) load1(R0, 2, i);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 8; ++i) read1(0, 0, A0, B0, i);
  int s = 0;
  for (; s + 1 < nsteps; s += 2) {  // two steps per trip, so the register sets stay static
    step(s, R1);
    step(s + 1, R0);
  }
  if (s < nsteps) step(s, R1);

  // Accumulator element e of lane l: column l%32, row 8(e/4) + 4(l/32) + e%4.
  // (One output pointer and one format flag, chosen before the loop: three
  // store paths inside it make the compiler hoist per-element addresses and
  // spill.)
  const bool full = m0 + 256 <= M && n0 + 256 <= N;
  // (The slab offset is formed in unsigned 32-bit pieces: a 64-bit copy of
  // ldy shared with the element addresses below turns each of them into a
  // full 64 x 64-bit multiply.)
  void* const Yo = part ? static_cast<void*>(part + (size_t)(blockIdx.y * (unsigned)M) * (unsigned)ldy) : Y;
  const int obf16 = part ? 0 : y_bf16;
  if (full && ldy < kFastStoreMaxLdy) {
    store_wave_tile(acc,
                    static_cast<char*>(Yo) + ((size_t)(unsigned)(m0 + 128 * wm) * (unsigned)ldy +
                                              (unsigned)(n0 + 128 * wn)) * (obf16 ? 2u : 4u),
                    ldy, obf16);
    return;
  }
#pragma unroll
  for (int a = 0; a < TI; ++a)
#pragma unroll
    for (int b = 0; b < TJ; ++b) {
      const int col = n0 + 128 * wn + 32 * b + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = m0 + 128 * wm + 32 * a + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (full || (row < M && col < N)) {
          if (obf16)
            static_cast<uint16_t*>(Yo)[(size_t)row * ldy + col] = f32_to_bf16_bits(acc[a][b][e]);
          else
            static_cast<float*>(Yo)[(size_t)row * ldy + col] = acc[a][b][e];
        }
      }
    }
}

// ---- 256 x 128 tile, one wave per SIMD ------------------------------------
// The 256 x 256 kernel's scheme on half the columns: four waves in a 2 x 2
// grid, each owning a 128 x 64 sub-tile (8 MFMA accumulators), so a 16-deep
// K slice is 8 MFMAs against 6 fragment reads.  A K step is four blocks of 8
// MFMA slots:
//   slices 0-1  fragment reads of the next slice at slots 0-5; the next step's
//               X rows written on odd slots (bf16 W: x0-x3, x4-x7; packed W:
//               two per slice, between the dequantized W writes at slots 3
//               and 7), its weight group dequantized a quarter of 8 columns
//               per slot (packed W)
//   slice 2     reads; the rest of the writes (bf16 W: w0-w3; packed W: x4-x7)
//   barrier
//   slice 3     reads of slice 0 of the next step
// with each global load of step + 3 issued one slot after the write that
// frees its register.  The MFMA chain of every output is the same as in the
// other kernels, hence the same bits.  K must be a multiple of 64 (shapes
// with a K tail take the general kernel).  Against the general kernel's
// 256 x 128 tiles (16 or 8 waves, the compiler's schedule), measured on MI355X
// with the same bits: Gemma3-4B o 41.6 -> 38.2 us (Q4NX weights), the 4B
// gate/up remainder 50.2 -> 44.7 us and the 27B o remainder 72.4 -> 55.1 us
// (bf16 weights), an MXFP4-variant 4B q/k/v product 54.9 -> 44.5 us.
constexpr int kW128LdsBytes = 2 * (256 + 128) * kLdsStride * 2;  // two stages of X (256 rows) and W (128 rows)

template <int WF>
struct Wide128Regs {
  u32x4 x[8];
  u32x4 q;
  uint32_t s, m;
};
template <>
struct Wide128Regs<kWBf16> {
  u32x4 x[8];
  u32x4 w[4];
};

template <int WF>
__global__ __launch_bounds__(kWideThreads) void gemm256x128_kernel(const uint16_t* __restrict__ X,
                                                                   const uint8_t* __restrict__ wsrc,
                                                                   void* __restrict__ Y, int M, int N, int K, int ldy,
                                                                   int KB, int NS, int tiles_n, int y_bf16) {
  constexpr int TI = 4, TJ = 2;
  extern __shared__ __attribute__((aligned(16))) uint16_t gl[];
  uint16_t* const xs0 = gl;                          // [2][256][72]
  uint16_t* const ws0 = gl + 2 * 256 * kLdsStride;   // [2][128][72]

  int bm, bn;
  gemm_tile_of(blockIdx.x, gridDim.x, tiles_n, bm, bn);
  const int m0 = bm * 256, n0 = bn * 128;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  const int rows_x = min(256, M - m0);
  const __amdgpu_buffer_rsrc_t rsx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(X + (size_t)m0 * K), (short)0, rows_x * K * 2, 0x00020000);
  constexpr bool WQ4 = WF != kWBf16;
  constexpr int kBB = wblock_bytes<WF>();
  const int s0 = n0 >> 5, nst = min(4, NS - s0), rows_w = min(128, N - n0);
  const __amdgpu_buffer_rsrc_t rsw =
      WQ4 ? __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(wsrc + (size_t)s0 * KB * kBB), (short)0,
                                              nst * KB * kBB, 0x00020000)
          : __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(wsrc + (size_t)n0 * K * 2), (short)0,
                                              rows_w * K * 2, 0x00020000);
  constexpr int kLoads = WF == kWQ4NX ? 11 : WF == kWMX ? 10 : 12;

  const int c8 = tid & 7, half = tid & 1;
  int vx[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) vx[i] = (min((tid >> 3) + 32 * i, rows_x - 1) * K + 8 * c8) * 2;
  int vq = 0, vs = 0, vw[4];
  if constexpr (WQ4) {
    const int r = tid >> 1;
    const int st = min(r >> 5, nst - 1), rr = r & 31;
    vq = st * KB * kBB + 128 * rr + 16 * half;
    vs = st * KB * kBB + kCodeBytes + (WF == kWMX ? 1 : 2) * (8 * rr + half);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) vw[i] = (min((tid >> 3) + 32 * i, rows_w - 1) * K + 8 * c8) * 2;
  }
  const int nsteps = K / kBK;

  f32x16 acc[TI][TJ];
#pragma unroll
  for (int a = 0; a < TI; ++a)
#pragma unroll
    for (int b = 0; b < TJ; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.0f;

  // Global load i of step t (clamped to the last step) into R.
  auto load1 = [&](Wide128Regs<WF>& R, int t, int i) {
    const int k0 = min(t, nsteps - 1) * kBK;
    const int sq = (k0 >> 8) * kBB + 16 * ((k0 & 255) >> 5);
    const int ss = (k0 >> 8) * kBB + (WF == kWMX ? 1 : 2) * ((k0 & 255) >> 5);
    if (i < 8) {
      R.x[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsx, vx[i], 2 * k0, 0));
      return;
    }
    if constexpr (!WQ4) {
      R.w[i - 8] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsw, vw[i - 8], 2 * k0, 0));
    } else if (i == 8) {
      R.q = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsw, vq + sq, 0, kNtLoad));
    } else if (i == 9) {
      if constexpr (WF == kWMX)
        R.s = __builtin_amdgcn_raw_buffer_load_b8(rsw, vs + ss, 0, kNtLoad);
      else
        R.s = __builtin_amdgcn_raw_buffer_load_b16(rsw, vs + ss, 0, kNtLoad);
    } else {
      R.m = __builtin_amdgcn_raw_buffer_load_b16(rsw, vs + ss + kScaleBytes, 0, kNtLoad);
    }
  };
  auto xs_row = [&](int st) { return xs0 + st * 256 * kLdsStride + (tid >> 3) * kLdsStride + 8 * c8; };
  auto ws_row = [&](int st) { return ws0 + st * 128 * kLdsStride + (tid >> 1) * kLdsStride + kGroup * half; };
  // Fragment i of K slice kq, in first-use order A0, B0, B1, A1, A2, A3.
  const int fa = (128 * wm + (lane & 31)) * kLdsStride + 8 * (lane >> 5);
  const int fb = (64 * wn + (lane & 31)) * kLdsStride + 8 * (lane >> 5);
  auto read1 = [&](int st, int kq, bf16x8 (&A)[TI], bf16x8 (&B)[TJ], int i) {
    const uint16_t* xs = xs0 + st * 256 * kLdsStride + fa + 16 * kq;
    const uint16_t* ws = ws0 + st * 128 * kLdsStride + fb + 16 * kq;
    if (i == 0) A[0] = *reinterpret_cast<const bf16x8*>(xs);
    else if (i <= 2) B[i - 1] = *reinterpret_cast<const bf16x8*>(ws + 32 * (i - 1) * kLdsStride);
    else A[i - 2] = *reinterpret_cast<const bf16x8*>(xs + 32 * (i - 2) * kLdsStride);
  };
  auto mma1 = [&](const bf16x8 (&A)[TI], const bf16x8 (&B)[TJ], int i) {
    acc[i >> 1][i & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(A[i >> 1], B[i & 1], acc[i >> 1][i & 1], 0, 0, 0);
  };
  // The thread's weight group of the next step dequantized piece by piece.
  GroupDequant<WF> gdq;
  auto wpiece = [&](const Wide128Regs<WF>& R, int st, int p) {
    if constexpr (WQ4) gdq.piece(R.q, R.s, WF == kWMX ? 0u : R.m, p, ws_row(st));
  };
  auto xwrite = [&](const Wide128Regs<WF>& R, uint16_t* xsn, int k) {
    *reinterpret_cast<u32x4*>(xsn + 32 * k * kLdsStride) = R.x[k];
  };
  auto wwrite = [&](const Wide128Regs<WF>& R, int st, int k) {
    if constexpr (!WQ4)
      *reinterpret_cast<u32x4*>(xs0 + 2 * 256 * kLdsStride + st * 128 * kLdsStride +
                                ((tid >> 3) + 32 * k) * kLdsStride + 8 * c8) = R.w[k];
  };

  bf16x8 A0[TI], B0[TJ], A1[TI], B1[TJ];
  // Work of slot i of slice sl besides the MFMA and the fragment read: the
  // stage writes of step s+1 (from Rs) and the loads of step s+3 (into Rs).
  auto side = [&](Wide128Regs<WF>& Rs, uint16_t* xsn, int nxt, int s, int sl, int i) {
    if constexpr (!WQ4) {
      // writes: slice 0 x0-x3, slice 1 x4-x7, slice 2 w0-w3 on odd slots;
      // load k one slot after write k (slot 0 of the next slice after slot 7)
      if (sl < 3 && (i & 1)) {
        const int k = 4 * sl + (i >> 1);
        if (k < 8) xwrite(Rs, xsn, k);
        else wwrite(Rs, nxt, k - 8);
      }
      if (!(i & 1)) {
        const int k = i == 0 ? 4 * sl - 1 : 4 * sl + (i >> 1) - 1;  // the write one slot back
        if (k >= 0 && k < 12 && !(sl == 3 && i > 0)) load1(Rs, s + 3, k);
      }
    } else {
      // dequant pieces 0-7 in slice 0, 8-15 in slice 1 (W writes at slots 3
      // and 7); X writes: slice 0 slots 1, 5; slice 1 slots 1, 5; slice 2
      // odd slots; loads: x one slot after its write, the scale (and offset)
      // after piece 0 consumed them, the codes in slice 2 after piece 15.
      if (sl < 2) wpiece(Rs, nxt, 8 * sl + i);
      int kx = -1;
      if (sl < 2 && (i == 1 || i == 5)) kx = 2 * sl + (i >> 2);
      if (sl == 2 && (i & 1)) kx = 4 + (i >> 1);
      if (kx >= 0) xwrite(Rs, xsn, kx);
      int kl = -1;
      if (sl < 2 && (i == 2 || i == 6)) kl = 2 * sl + (i >> 2);
      if (sl == 2 && !(i & 1) && i > 0) kl = 4 + (i >> 1) - 1;
      if (sl == 3 && i == 0) kl = 7;
      if (kl >= 0) load1(Rs, s + 3, kl);
      if (sl == 0 && i == 4) load1(Rs, s + 3, 9);                         // scale
      if (WF == kWQ4NX && sl == 0 && i == 6) load1(Rs, s + 3, 10);        // offset
      if (sl == 2 && i == 0) load1(Rs, s + 3, 8);                         // codes
    }
  };
  auto step = [&](int s, Wide128Regs<WF>& Rs) {
    const int cur = s & 1, nxt = cur ^ 1;
    uint16_t* xsn = xs_row(nxt);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      mma1(A0, B0, i);
      if (i < 6) read1(cur, 1, A1, B1, i);
      side(Rs, xsn, nxt, s, 0, i);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      mma1(A1, B1, i);
      if (i < 6) read1(cur, 2, A0, B0, i);
      side(Rs, xsn, nxt, s, 1, i);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      mma1(A0, B0, i);
      if (i < 6) read1(cur, 3, A1, B1, i);
      side(Rs, xsn, nxt, s, 2, i);
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      mma1(A1, B1, i);
      if (i < 6) read1(nxt, 0, A0, B0, i);
      side(Rs, xsn, nxt, s, 3, i);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  Wide128Regs<WF> R0, R1;
#pragma unroll
  for (int i = 0; i < kLoads; ++i) load1(R0, 0, i);
#pragma unroll
  for (int i = 0; i < kLoads; ++i) load1(R1, 1, i);
  {
    uint16_t* xs = xs_row(0);
#pragma unroll
    for (int i = 0; i < 8; ++i) xwrite(R0, xs, i);
    if constexpr (WF == kWMX) {
      const float Xs = e8m0_f32(R0.s);
#pragma unroll
      for (int u = 0; u < 4; ++u) *reinterpret_cast<u32x4*>(ws_row(0) + 8 * u) = mx8_bf16(R0.q[u], Xs);
    } else if constexpr (WQ4) {
      const float d512 = bf16_to_f32(R0.s) * 512.0f, m = bf16_to_f32(R0.m);
#pragma unroll
      for (int u = 0; u < 4; ++u) *reinterpret_cast<u32x4*>(ws_row(0) + 8 * u) = dequant8_bf16(R0.q[u], d512, m);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) wwrite(R0, 0, i);
    }
  }
#pragma unroll
  for (int i = 0; i < kLoads; ++i) load1(R0, 2, i);
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 6; ++i) read1(0, 0, A0, B0, i);
  int s = 0;
  for (; s + 1 < nsteps; s += 2) {
    step(s, R1);
    step(s + 1, R0);
  }
  if (s < nsteps) step(s, R1);

  const bool full = m0 + 256 <= M && n0 + 128 <= N;
  if (full && ldy < kFastStoreMaxLdy) {
    store_wave_tile(acc,
                    static_cast<char*>(Y) + ((size_t)(unsigned)(m0 + 128 * wm) * (unsigned)ldy +
                                             (unsigned)(n0 + 64 * wn)) * (y_bf16 ? 2u : 4u),
                    ldy, y_bf16);
    return;
  }
#pragma unroll
  for (int a = 0; a < TI; ++a)
#pragma unroll
    for (int b = 0; b < TJ; ++b) {
      const int col = n0 + 64 * wn + 32 * b + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = m0 + 128 * wm + 32 * a + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (full || (row < M && col < N)) {
          if (y_bf16)
            static_cast<uint16_t*>(Y)[(size_t)row * ldy + col] = f32_to_bf16_bits(acc[a][b][e]);
          else
            static_cast<float*>(Y)[(size_t)row * ldy + col] = acc[a][b][e];
        }
      }
    }
}

// Sum of the split-K partial products part[0..ks-1][M][N] (row stride N), in
// segment order, to Y (row stride ldy) in float32 or bf16.  Thread t handles
// four consecutive columns of one row.  With vec (N and ldy multiples of 4,
// Y 16-byte aligned) a full quad is read as one 16-byte load per segment --
// every segment's load issued before the adds -- and written as one store;
// the order of the adds, hence every bit, is that of the scalar path.
__global__ __launch_bounds__(256) void splitk_sum_kernel(const float* __restrict__ part, int ks, int M, int N,
                                                         void* __restrict__ Y, int64_t ldy, int y_bf16, int vec) {
  const int q = (N + 3) >> 2;  // column quads per row
  const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (id >= (int64_t)M * q) return;
  const int row = (int)(id / q), col = (int)(id - (int64_t)row * q) * 4;
  const int64_t MN = (int64_t)M * N;
  const float* p = part + (int64_t)row * N + col;
  if (vec && col + 3 < N) {
    f32x4 seg[kMaxSplit];
#pragma unroll
    for (int s = 0; s < kMaxSplit; ++s)
      if (s < ks) seg[s] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + s * MN));
    f32x4 v = seg[0];
#pragma unroll
    for (int s = 1; s < kMaxSplit; ++s)
      if (s < ks) v += seg[s];
    if (y_bf16) {
      typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
      *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(Y) + row * ldy + col) =
          (u32x2){pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
    } else {
      *reinterpret_cast<f32x4*>(static_cast<float*>(Y) + row * ldy + col) = v;
    }
    return;
  }
  float v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = col + j < N ? p[j] : 0.0f;
  for (int s = 1; s < ks; ++s)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (col + j < N) v[j] += p[s * MN + j];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (col + j >= N) break;
    if (y_bf16)
      static_cast<uint16_t*>(Y)[row * ldy + col + j] = f32_to_bf16_bits(v[j]);
    else
      static_cast<float*>(Y)[row * ldy + col + j] = v[j];
  }
}

// ---- general tiles, two waves per SIMD --------------------------------------
// Workgroup tile BM (tokens) x BN (outputs) for the shapes the 256 x 256 and
// 256 x 128 hand-scheduled tiles do not serve (128 x 128 and 128 x 64 tiles,
// 256 x 128 tiles with a K tail).  WAVES_M x WAVES_N waves; each owns a (BM/WAVES_M) x
// (BN/WAVES_N) sub-tile.  LDS holds two stages of the X tile and of the
// dequantized W tile; a K step runs the MFMAs of step k from one stage while
// the same waves dequantize step k+1 into the other, with the raw global data
// of step k+1 loaded into registers two steps earlier.  One workgroup barrier
// per K step.
template <int BM, int BN, int WAVES_M, int WAVES_N>
struct GemmCfg {
  static constexpr int kThreads = 64 * WAVES_M * WAVES_N;
  static constexpr int kWTM = BM / WAVES_M, kWTN = BN / WAVES_N;
  static constexpr int kTI = kWTM / 32, kTJ = kWTN / 32;
  static constexpr int kXChunks = BM * (kBK / 8) / kThreads;   // 16-byte X chunks per thread per step
  // Weight groups per step and per thread (threads past the step's groups --
  // whole waves, since BN * 2 is a multiple of 64 -- dequantize none).
  static constexpr int kStepGroups = BN * (kBK / kGroup);
  static constexpr int kWGroups = (kStepGroups + kThreads - 1) / kThreads;
  static constexpr int kWChunks = BN * (kBK / 8) / kThreads;   // 16-byte chunks of a bf16 W tile
  static constexpr int kLdsElems = 2 * (BM + BN) * kLdsStride;
  static_assert(kXChunks >= 1 && kWGroups >= 1, "tile too small for the thread count");
  static_assert(kTI >= 1 && kTJ >= 1, "wave tile below 32 x 32");
};

// Raw global data of one K step held by one thread: its X chunks and either
// the codes / scale / offset of its weight groups or its bf16 W chunks.
template <int XC, int WG, int WC>
struct GemmRegs {
  u32x4 x[XC];
  u32x4 q[WG];
  uint32_t s[WG], m[WG];
  u32x4 w[WC];
};

// WF: W is a packed Q4NX or MXFP4-variant matrix (blob), or bf16 [N][K].
template <int BM, int BN, int WAVES_M, int WAVES_N, int WF>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void gemm_kernel(
    const uint16_t* __restrict__ X, const uint8_t* __restrict__ blob, void* __restrict__ Y, int M, int N, int K,
    int ldy, int KB, int NS, int tiles_n, int y_bf16) {
  constexpr bool WQ4 = WF != kWBf16;  // packed weights
  using C = GemmCfg<BM, BN, WAVES_M, WAVES_N>;
  using Regs = GemmRegs<C::kXChunks, WQ4 ? C::kWGroups : 1, WQ4 ? 1 : C::kWChunks>;
  const uint16_t* const Wb = reinterpret_cast<const uint16_t*>(blob);
  extern __shared__ __attribute__((aligned(16))) uint16_t gl[];
  uint16_t* xs0 = gl;                              // [2][BM][72]
  uint16_t* ws0 = gl + 2 * BM * kLdsStride;        // [2][BN][72]

  int bm, bn;
  gemm_tile_of(blockIdx.x, gridDim.x, tiles_n, bm, bn);
  const int m0 = bm * BM, n0 = bn * BN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;

  f32x16 acc[C::kTI][C::kTJ];
#pragma unroll
  for (int a = 0; a < C::kTI; ++a)
#pragma unroll
    for (int b = 0; b < C::kTJ; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.0f;

  // Global loads of step k0 into registers.  Row and column indices are
  // clamped so every address is inside the operands; the values that belong
  // outside the matrices are zeroed only when the step is stored, so nothing
  // here waits for the loads to return.
  auto load_step = [&](Regs& R, int k0) {
#pragma unroll
    for (int i = 0; i < C::kXChunks; ++i) {
      const int ch = tid + i * C::kThreads;       // chunk: row ch/8, columns 8(ch%8)..+7
      const int r = ch >> 3, kk = k0 + 8 * (ch & 7);
      R.x[i] = *reinterpret_cast<const u32x4*>(X + (size_t)min(m0 + r, M - 1) * K + min(kk, K - 8));
    }
    if constexpr (!WQ4) {
#pragma unroll
      for (int i = 0; i < C::kWChunks; ++i) {
        const int ch = tid + i * C::kThreads;     // chunk: W row ch/8, columns 8(ch%8)..+7
        const int r = ch >> 3, kk = k0 + 8 * (ch & 7);
        R.w[i] = *reinterpret_cast<const u32x4*>(Wb + (size_t)min(n0 + r, N - 1) * K + min(kk, K - 8));
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < C::kWGroups; ++i) {
      const int gi = tid + i * C::kThreads;       // group: row gi/2, half gi%2 of the K step
      if (C::kStepGroups % C::kThreads != 0 && gi >= C::kStepGroups) break;  // wave-uniform
      const int r = gi >> 1, gk = min(k0 + kGroup * (gi & 1), K - kGroup);
      const int gn = n0 + r, rr = gn & 31;
      const int j = gk >> 8, c = (gk & 255) >> 5;
      const uint8_t* blk = blob + ((size_t)min(gn >> 5, NS - 1) * KB + j) * wblock_bytes<WF>();
      R.q[i] = load_codes(blk + 128 * rr + 16 * c);
      if constexpr (WF == kWMX) {
        R.s[i] = load_u8(blk + kCodeBytes + 8 * rr + c);
      } else {
        R.s[i] = load_u16(blk + kCodeBytes + 2 * (8 * rr + c));
        R.m[i] = load_u16(blk + kCodeBytes + kScaleBytes + 2 * (8 * rr + c));
      }
    }
  };

  // Zero what lies outside the matrices, dequantize the weight groups (Eq. 3
  // in float32, rounded to bf16) and write X and W of step k0 to LDS stage st.
  auto store_step = [&](const Regs& R, int st, int k0) {
    uint16_t* xs = xs0 + st * BM * kLdsStride;
    uint16_t* ws = ws0 + st * BN * kLdsStride;
#pragma unroll
    for (int i = 0; i < C::kXChunks; ++i) {
      const int ch = tid + i * C::kThreads;
      const bool ok = m0 + (ch >> 3) < M && k0 + 8 * (ch & 7) < K;
      *reinterpret_cast<u32x4*>(xs + (ch >> 3) * kLdsStride + 8 * (ch & 7)) = ok ? R.x[i] : (u32x4){0u, 0u, 0u, 0u};
    }
    if constexpr (!WQ4) {
#pragma unroll
      for (int i = 0; i < C::kWChunks; ++i) {
        const int ch = tid + i * C::kThreads;
        const bool ok = n0 + (ch >> 3) < N && k0 + 8 * (ch & 7) < K;
        *reinterpret_cast<u32x4*>(ws + (ch >> 3) * kLdsStride + 8 * (ch & 7)) = ok ? R.w[i] : (u32x4){0u, 0u, 0u, 0u};
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < C::kWGroups; ++i) {
      const int gi = tid + i * C::kThreads;
      if (C::kStepGroups % C::kThreads != 0 && gi >= C::kStepGroups) break;  // wave-uniform
      const bool ok = ((n0 + (gi >> 1)) >> 5) < NS && k0 + kGroup * (gi & 1) < K;
      const u32x4 q = ok ? R.q[i] : (u32x4){0u, 0u, 0u, 0u};
      if constexpr (WF == kWMX) {
        const float Xs = ok ? e8m0_f32(R.s[i]) : 0.0f;
        u32x4* wd = reinterpret_cast<u32x4*>(ws + (gi >> 1) * kLdsStride + kGroup * (gi & 1));
#pragma unroll
        for (int v = 0; v < 4; ++v) wd[v] = mx8_bf16(q[v], Xs);
        continue;
      }
      const float d512 = ok ? bf16_to_f32(R.s[i]) * 512.0f : 0.0f, m = ok ? bf16_to_f32(R.m[i]) : 0.0f;
      u32x4* wd = reinterpret_cast<u32x4*>(ws + (gi >> 1) * kLdsStride + kGroup * (gi & 1));
#pragma unroll
      for (int v = 0; v < 4; ++v) wd[v] = dequant8_bf16(q[v], d512, m);
    }
  };

  // The MFMAs of one K step from LDS stage st.
  auto mma_step = [&](int st) {
    const uint16_t* xs = xs0 + st * BM * kLdsStride;
    const uint16_t* ws = ws0 + st * BN * kLdsStride;
#pragma unroll
    for (int kq = 0; kq < kBK / 16; ++kq) {
      const int kk = kq * 16 + 8 * (lane >> 5);
      bf16x8 af[C::kTI], bfr[C::kTJ];
#pragma unroll
      for (int a = 0; a < C::kTI; ++a)
        af[a] = *reinterpret_cast<const bf16x8*>(xs + (C::kWTM * wm + 32 * a + (lane & 31)) * kLdsStride + kk);
#pragma unroll
      for (int b = 0; b < C::kTJ; ++b)
        bfr[b] = *reinterpret_cast<const bf16x8*>(ws + (C::kWTN * wn + 32 * b + (lane & 31)) * kLdsStride + kk);
#pragma unroll
      for (int a = 0; a < C::kTI; ++a)
#pragma unroll
        for (int b = 0; b < C::kTJ; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    }
  };

  const int nsteps = (K + kBK - 1) / kBK;
  Regs R0, R1;
  load_step(R0, 0);
  store_step(R0, 0, 0);
  load_step(R0, kBK);
  load_step(R1, 2 * kBK);
  __syncthreads();
  int ks = 0;
  // Steady state, two steps per trip so the register sets stay static.
  for (; ks + 2 < nsteps; ks += 2) {
    mma_step(0);
    store_step(R0, 1, (ks + 1) * kBK);
    // Unconditional (addresses are clamped; data past the last step is never
    // stored), so the wait-count bookkeeping sees the same load order on every
    // trip and waits only for the register set being consumed.
    load_step(R0, (ks + 3) * kBK);
    __syncthreads();
    mma_step(1);
    store_step(R1, 0, (ks + 2) * kBK);
    load_step(R1, (ks + 4) * kBK);
    __syncthreads();
  }
  // Tail: one or two steps left; step ks+1 (if any) is in R0.
  if (ks + 1 < nsteps) {
    mma_step(ks & 1);
    store_step(R0, (ks + 1) & 1, (ks + 1) * kBK);
    __syncthreads();
    ++ks;
  }
  mma_step(ks & 1);

  if (m0 + BM <= M && n0 + BN <= N && ldy < kFastStoreMaxLdy) {
    store_wave_tile(acc,
                    static_cast<char*>(Y) + ((size_t)(unsigned)(m0 + C::kWTM * wm) * (unsigned)ldy +
                                             (unsigned)(n0 + C::kWTN * wn)) * (y_bf16 ? 2u : 4u),
                    ldy, y_bf16);
    return;
  }
  // Accumulator element e of lane l: column l%32, row 8(e/4) + 4(l/32) + e%4.
#pragma unroll
  for (int a = 0; a < C::kTI; ++a)
#pragma unroll
    for (int b = 0; b < C::kTJ; ++b) {
      const int col = n0 + C::kWTN * wn + 32 * b + (lane & 31);
      if (col >= N) continue;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = m0 + C::kWTM * wm + 32 * a + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        if (row < M) {
          if (y_bf16)
            static_cast<uint16_t*>(Y)[(size_t)row * ldy + col] = f32_to_bf16_bits(acc[a][b][e]);
          else
            static_cast<float*>(Y)[(size_t)row * ldy + col] = acc[a][b][e];
        }
      }
    }
}

// ---- launch planning ----------------------------------------------------------
// Tile shapes: 0 = 256 x 256 (gemm256_kernel; the general kernel past
// kWideMaxK), 1 = 256 x 128 (gemm256x128_kernel; the general kernel with a K
// tail or past kWideMaxK), 2 = 128 x 128, 3 = 128 x 64 (the general kernel).
// The round costs below were measured with the general kernel's 256 x 128
// tiles; the one-wave-per-SIMD form is faster on the Gemma3 shapes it serves,
// which only favours the plans that use it.
struct GemmTile {
  int bm, bn;
  float round_cost;  // time of one full round (a tile on every CU), relative to shape 0
};
// Round costs measured on MI355X for the Gemma3 prefill projections (K = 5376).
constexpr GemmTile kGemmTiles[4] = {{256, 256, 1.0f}, {256, 128, 0.68f}, {128, 128, 0.52f}, {128, 64, 0.38f}};

// A rectangle of the output computed by one launch (ks > 1: by ks K segments
// of the 256 x 256 kernel and a second launch that adds their partials).
struct GemmRegion {
  int tile;
  int64_t m0, n0, M, N;
  int ks;
};

// Split K.  With a caller workspace, a 256 x 256 launch may run every tile as
// ks K segments on ks workgroups that write float32 partial products, which a
// second launch adds in segment order (deterministic).  It pays where a long
// K meets few tiles (Gemma3 down projections).  Split plans are costed in the
// planner's unit, a round of 256 x 256 tiles at the full K, through a time
// model fitted on MI355X: such a round over K columns takes about
// 40 + 0.0226 K us, and the sum streams its operands at about 5 TB/s after a
// ~5 us launch.
constexpr double kRoundFixedUs = 40.0, kRoundPerKUs = 0.0226;
constexpr double kSumLaunchUs = 5.0, kSumBytesPerUs = 5.0e6;
// (The round costs and this model were fitted before the buffer-store
// epilogue took 6-10 us off every round.  A refit from single full rounds,
// about 16 + 0.0237 K us and costs 1 : 0.65 : 0.40 : 0.32, picks worse plans
// for partly filled launches -- e.g. a two-shape split of 4096 x 2560 x 2048
// that runs 23% slower than one partial round of 256 x 256 tiles -- while
// the plans chosen here measure within 2% of the best forced plan on every
// Gemma3 prefill product, so they are kept.)
constexpr int kMinSegmentSteps = 8;

static double round_us(int64_t K) { return kRoundFixedUs + kRoundPerKUs * (double)K; }

// K steps per segment when K is split into ks non-empty segments of at least
// kMinSegmentSteps steps each; 0 if it cannot be.
static int split_steps(int64_t K, int ks) {
  if (ks < 2 || K >= kWideMaxK) return 0;
  const int64_t nsteps = ceil_div(K, kBK), per = ceil_div(nsteps, ks);
  return (per >= kMinSegmentSteps && (ks - 1) * per < nsteps) ? (int)per : 0;
}

static int device_cus() { return current_device_cus(); }

// Chooses one launch, or two launches over a split of the rows or columns,
// minimising the estimated time: sum over launches of (rounds of tiles on the
// CUs) x (round cost of the tile shape), plus a small cost per extra launch.
// A launch whose last round is only partly filled still pays a whole round,
// so a shape with 336 256x256 tiles on 256 CUs is better done as one full
// round of 256 x 256 tiles and the rest in smaller tiles.  With split_ok, the
// whole product or the second region may also be split along K.
static int gemm_plan(int64_t M, int64_t N, int64_t K, int cus, bool split_ok, GemmRegion (&plan)[2],
                     double* est_us = nullptr) {
  const auto rounds = [&](int t, int64_t m, int64_t n) {
    return (double)ceil_div(ceil_div(m, kGemmTiles[t].bm) * ceil_div(n, kGemmTiles[t].bn), cus);
  };
  // Cost of an (m x n) region as ks K segments of 256 x 256 tiles plus the sum.
  const auto split_cost = [&](int64_t m, int64_t n, int ks) {
    const int per = split_steps(K, ks);
    if (!split_ok || per == 0) return 1e300;
    const double r = (double)ceil_div(ceil_div(m, 256) * ceil_div(n, 256) * ks, cus);
    const double sum_us = kSumLaunchUs + (4.0 * ks + 4.0) * (double)m * (double)n / kSumBytesPerUs;
    return (r * round_us((int64_t)per * kBK) + sum_us) / round_us(K);
  };
  double best = 1e300;
  int count = 0;
  for (int ks = 2; ks <= kMaxSplit; ++ks) {
    const double c = split_cost(M, N, ks);
    if (c < best) {
      best = c;
      plan[0] = {0, 0, 0, M, N, ks};
      count = 1;
    }
  }
  for (int a = 0; a < 4; ++a) {
    const double c1 = rounds(a, M, N) * kGemmTiles[a].round_cost;
    if (c1 < best) {
      best = c1;
      plan[0] = {a, 0, 0, M, N, 1};
      count = 1;
    }
    const int64_t tm = ceil_div(M, kGemmTiles[a].bm), tn = ceil_div(N, kGemmTiles[a].bn);
    const int64_t full = (tm * tn) / cus;  // whole rounds of shape a
    if (full < 1) continue;
    for (int dir = 0; dir < 2; ++dir) {
      // Largest leading block of rows (dir 0) or columns (dir 1) whose tiles
      // fit in the whole rounds; the rest goes to a smaller shape.
      const int64_t split = dir == 0 ? (full * cus / tn) * kGemmTiles[a].bm : (full * cus / tm) * kGemmTiles[a].bn;
      if (split <= 0 || split >= (dir == 0 ? M : N)) continue;
      const int64_t ma = dir == 0 ? split : M, na = dir == 0 ? N : split;
      const int64_t mb = dir == 0 ? M - split : M, nb = dir == 0 ? N : N - split;
      for (int b = a + 1; b < 4; ++b) {
        const double c2 = rounds(a, ma, na) * kGemmTiles[a].round_cost +
                          rounds(b, mb, nb) * kGemmTiles[b].round_cost + 0.02 + 0.001 * dir;
        if (c2 < best) {
          best = c2;
          plan[0] = {a, 0, 0, ma, na, 1};
          plan[1] = {b, dir == 0 ? split : 0, dir == 0 ? 0 : split, mb, nb, 1};
          count = 2;
        }
      }
      for (int ks = 2; ks <= kMaxSplit; ++ks) {
        const double c2 = rounds(a, ma, na) * kGemmTiles[a].round_cost + split_cost(mb, nb, ks) + 0.02 + 0.001 * dir;
        if (c2 < best) {
          best = c2;
          plan[0] = {a, 0, 0, ma, na, 1};
          plan[1] = {0, dir == 0 ? split : 0, dir == 0 ? 0 : split, mb, nb, ks};
          count = 2;
        }
      }
    }
  }
  if (est_us) *est_us = best * round_us(K);
  return count;
}

// Workspace bytes a plan needs: the regions run one after the other on one
// stream, so they share it.
static size_t plan_work_bytes(const GemmRegion* plan, int count) {
  size_t b = 0;
  for (int i = 0; i < count; ++i)
    if (plan[i].ks > 1) b = std::max(b, (size_t)plan[i].ks * (size_t)plan[i].M * (size_t)plan[i].N * sizeof(float));
  return b;
}

// Dequantize, then multiply.  The fused kernel dequantizes every weight once
// per row of output tiles (16 times at M = 4096).  With a workspace that holds
// W in bf16, a Q4NX product can dequantize each weight once instead (the
// dequant kernel streams at ~5.5 TB/s) and run the same plan on the bf16
// weights: the same bf16 values, the same MFMA chains and partial sums, so
// the same bits.  The fused kernel's extra work is Eq. 3 inside the K loop:
// measured on MI355X it adds about a fifth of the K-loop time of the
// 256 x 256 kernel (1.19-1.26 x the bf16 product's time on the Gemma3 4B and
// 27B products) and about a seventh for the smaller tiles of the general
// kernel, so the two-phase route is taken when the dequantization pass is
// estimated below that share of the planned K-loop time: every Gemma3 27B
// product at M = 4096, the 4B gate/up and down products at M = 2048, not the
// 4B q/k/v and o products (short K, smaller tiles) nor M <= 1024.  (The
// MXFP4 variant's conversion is cheap enough that the fused kernel runs at
// the bf16 speed.)
constexpr double kDequantLaunchUs = 3.0, kDequantBytesPerUs = 5.5e6;
constexpr double kFusedExtraWide = 0.20, kFusedExtraSmall = 0.14;

struct GemmChoice {
  GemmRegion plan[2];
  int count;
  bool two_phase;
  size_t w_bytes;     // bf16 W at the start of the workspace (two-phase only)
  size_t part_bytes;  // split-K partial products after it
};

static GemmChoice gemm_choose(int wf, int64_t M, int64_t N, int64_t K, bool have_work) {
  GemmChoice c{};
  double est_us = 0.0;
  c.count = gemm_plan(M, N, K, device_cus(), have_work, c.plan, &est_us);
  c.part_bytes = plan_work_bytes(c.plan, c.count);
  const double deq_us = kDequantLaunchUs + (kBlockBytes / (double)(kBlockRows * kBlockCols) + 2.0) * (double)N *
                                               (double)K / kDequantBytesPerUs;
  const double kloop_us = est_us * kRoundPerKUs * (double)K / round_us(K);
  const double extra = c.plan[0].tile == 0 ? kFusedExtraWide : kFusedExtraSmall;
  c.two_phase = have_work && wf == kWQ4NX && deq_us < extra * kloop_us;
  c.w_bytes = c.two_phase ? (size_t)ceil_div(N * K * 2, 256) * 256 : 0;
  return c;
}

template <int BM, int BN, int WAVES_M, int WAVES_N, int WF>
static q4nx_status launch_gemm(int64_t M, int64_t N, int64_t K, const uint16_t* X, const void* blob, void* Y,
                               int64_t ldy, int y_bf16, hipStream_t stream) {
  using Cfg = GemmCfg<BM, BN, WAVES_M, WAVES_N>;
  const int64_t tiles_n = ceil_div(N, BN), tiles_m = ceil_div(M, BM);
  const size_t lds = sizeof(uint16_t) * Cfg::kLdsElems;
  auto kern = gemm_kernel<BM, BN, WAVES_M, WAVES_N, WF>;
  static LdsReservation lds_res;  // LDS above 64 KiB, requested once per device
  if (!lds_res.ensure(reinterpret_cast<const void*>(kern), (int)lds))
    return fail(Q4NX_ERR_HIP, "q4nx_gemm: cannot reserve LDS");
  hipLaunchKernelGGL(kern, dim3((unsigned)(tiles_n * tiles_m)), dim3(Cfg::kThreads), lds, stream, X,
                     static_cast<const uint8_t*>(blob), Y, (int)M, (int)N, (int)K, (int)ldy,
                     (int)ceil_div(K, kBlockCols), (int)ceil_div(N, kBlockRows), (int)tiles_n, y_bf16);
  return Q4NX_OK;
}

template <bool KTAIL, int WF>
static q4nx_status launch_gemm256(int64_t M, int64_t N, int64_t K, const uint16_t* X, const void* blob, void* Y,
                                  int64_t ldy, int y_bf16, hipStream_t stream, int ks = 1, float* part = nullptr) {
  auto kern = gemm256_kernel<KTAIL, WF>;
  static LdsReservation lds_res;
  if (!lds_res.ensure(reinterpret_cast<const void*>(kern), kWideLdsBytes))
    return fail(Q4NX_ERR_HIP, "q4nx_gemm: cannot reserve LDS");
  const int64_t tiles_n = ceil_div(N, 256), tiles_m = ceil_div(M, 256);
  const int ksteps = ks > 1 ? split_steps(K, ks) : (int)ceil_div(K, kBK);
  hipLaunchKernelGGL(kern, dim3((unsigned)(tiles_n * tiles_m), (unsigned)ks), dim3(kWideThreads), kWideLdsBytes,
                     stream, X, static_cast<const uint8_t*>(blob), Y, (int)M, (int)N, (int)K, (int)ldy,
                     (int)ceil_div(K, kBlockCols), (int)ceil_div(N, kBlockRows), (int)tiles_n, y_bf16, ksteps,
                     ks > 1 ? part : nullptr);
  return Q4NX_OK;
}

template <int WF>
static q4nx_status launch_gemm256x128(int64_t M, int64_t N, int64_t K, const uint16_t* X, const void* blob, void* Y,
                                      int64_t ldy, int y_bf16, hipStream_t stream) {
  auto kern = gemm256x128_kernel<WF>;
  static LdsReservation lds_res;
  if (!lds_res.ensure(reinterpret_cast<const void*>(kern), kW128LdsBytes))
    return fail(Q4NX_ERR_HIP, "q4nx_gemm: cannot reserve LDS");
  const int64_t tiles_n = ceil_div(N, 128), tiles_m = ceil_div(M, 256);
  hipLaunchKernelGGL(kern, dim3((unsigned)(tiles_n * tiles_m)), dim3(kWideThreads), kW128LdsBytes, stream, X,
                     static_cast<const uint8_t*>(blob), Y, (int)M, (int)N, (int)K, (int)ldy,
                     (int)ceil_div(K, kBlockCols), (int)ceil_div(N, kBlockRows), (int)tiles_n, y_bf16);
  return Q4NX_OK;
}

// One region of the output: X rows m0.., W rows n0.. (strips n0/32.. of a
// packed matrix) and Y at (m0, n0) with row stride N, so each launch sees an
// ordinary smaller problem.
template <int WF>
static q4nx_status launch_region(const GemmRegion& r, int64_t N, int64_t K, const uint16_t* X, const void* w,
                                 void* Y, int y_bf16, hipStream_t stream, float* work) {
  const uint16_t* Xr = X + r.m0 * K;
  const void* Wr = WF != kWBf16
                       ? static_cast<const void*>(static_cast<const uint8_t*>(w) +
                                                  (r.n0 / kBlockRows) * ceil_div(K, kBlockCols) * wblock_bytes<WF>())
                       : static_cast<const void*>(static_cast<const uint16_t*>(w) + r.n0 * K);
  void* Yr = static_cast<uint8_t*>(Y) + (r.m0 * N + r.n0) * (y_bf16 ? 2 : 4);
  if (r.ks > 1) {
    // Partials [ks][r.M][r.N] in the workspace, then their sum into Y.
    const q4nx_status st = K % kBK != 0
                               ? launch_gemm256<true, WF>(r.M, r.N, K, Xr, Wr, Yr, r.N, y_bf16, stream, r.ks, work)
                               : launch_gemm256<false, WF>(r.M, r.N, K, Xr, Wr, Yr, r.N, y_bf16, stream, r.ks, work);
    if (st != Q4NX_OK) return st;
    const int64_t threads = r.M * ceil_div(r.N, 4);
    const int vec = r.N % 4 == 0 && N % 4 == 0 && aligned(Yr, 16);
    hipLaunchKernelGGL(splitk_sum_kernel, dim3((unsigned)ceil_div(threads, 256)), dim3(256), 0, stream, work, r.ks,
                       (int)r.M, (int)r.N, Yr, N, y_bf16, vec);
    return Q4NX_OK;
  }
  switch (r.tile) {
    case 0:
      if (K >= kWideMaxK) return launch_gemm<256, 256, 2, 4, WF>(r.M, r.N, K, Xr, Wr, Yr, N, y_bf16, stream);
      if (K % kBK != 0) return launch_gemm256<true, WF>(r.M, r.N, K, Xr, Wr, Yr, N, y_bf16, stream);
      return launch_gemm256<false, WF>(r.M, r.N, K, Xr, Wr, Yr, N, y_bf16, stream);
    case 1:
      if (K % kBK == 0 && K < kWideMaxK) return launch_gemm256x128<WF>(r.M, r.N, K, Xr, Wr, Yr, N, y_bf16, stream);
      // A K tail: the general kernel.  Q4NX weights as 16 waves of 32 x 64
      // (four per SIMD), which hide the dequantization in the tile loads
      // better than 8 waves of 64 x 64 (measured on MI355X: Gemma3 4B q/k/v
      // 56.8 -> 55.5 us, o 42.2 -> 39.2 us with K a multiple of 64); bf16 and
      // MXFP4-variant weights keep 8 waves (the 4B bf16 gate/up remainder ran
      // 2.6% slower with 16).  Same MFMA chains, same bits.
      if constexpr (WF == kWQ4NX) return launch_gemm<256, 128, 8, 2, WF>(r.M, r.N, K, Xr, Wr, Yr, N, y_bf16, stream);
      else return launch_gemm<256, 128, 4, 2, WF>(r.M, r.N, K, Xr, Wr, Yr, N, y_bf16, stream);
    case 2: return launch_gemm<128, 128, 2, 4, WF>(r.M, r.N, K, Xr, Wr, Yr, N, y_bf16, stream);
    default: return launch_gemm<128, 64, 2, 2, WF>(r.M, r.N, K, Xr, Wr, Yr, N, y_bf16, stream);
  }
}

static q4nx_status check_launch(const char* fn);

// Validation shared by the matrix-product entry points, then the planned
// launches (split along K only when a workspace is given).
template <int WF>
static q4nx_status gemm_entry(int64_t M, int64_t N, int64_t K, const uint16_t* d_X, const void* d_W, void* d_Y,
                              q4nx_dtype y_dtype, void* d_work, size_t work_bytes, hipStream_t stream,
                              const char* fn) {
  clear_error();
  if (q4nx_status st = check_shape(N, K, fn)) return st;
  if (M <= 0 || M > Q4NX_MAX_DIM) return fail(Q4NX_ERR_SHAPE, std::string(fn) + ": M must lie in 1..2^30");
  if (!d_X || !d_W || !d_Y) return fail(Q4NX_ERR_INVALID_ARG, std::string(fn) + ": NULL pointer");
  if (y_dtype != Q4NX_F32 && y_dtype != Q4NX_BF16)
    return fail(Q4NX_ERR_INVALID_ARG, std::string(fn) + ": unknown y_dtype");
  if (!aligned(d_X, 16) || !aligned(d_W, 16) || !aligned(d_Y, 16))
    return fail(Q4NX_ERR_ALIGNMENT, std::string(fn) + (WF != kWBf16 ? ": X, blob and Y need 16-byte alignment"
                                                                    : ": X, W and Y need 16-byte alignment"));
  if (M * N > (int64_t(1) << 40)) return fail(Q4NX_ERR_SHAPE, std::string(fn) + ": problem too large for one launch");
  if (d_work && !aligned(d_work, 16)) return fail(Q4NX_ERR_ALIGNMENT, std::string(fn) + ": work needs 16-byte alignment");
  const GemmChoice c = gemm_choose(WF, M, N, K, d_work != nullptr);
  if (c.w_bytes + c.part_bytes > work_bytes)
    return fail(Q4NX_ERR_BUFFER_TOO_SMALL, std::string(fn) + ": work_bytes < q4nx_gemm_workspace_size(...)");
  const int y_bf16 = y_dtype == Q4NX_BF16;
  float* part = reinterpret_cast<float*>(static_cast<uint8_t*>(d_work) + c.w_bytes);
  q4nx_status st = Q4NX_OK;
  if (c.two_phase) {
    const int64_t KB = ceil_div(K, kBlockCols), nblocks = ceil_div(N, kBlockRows) * KB;
    hipLaunchKernelGGL(dequant_kernel<kWQ4NX>, dim3((unsigned)std::min<int64_t>(nblocks, int64_t(1) << 20)),
                       dim3(256), 0, stream, static_cast<const uint8_t*>(d_W), N, K, KB, nblocks, d_work, 1);
    for (int i = 0; i < c.count && st == Q4NX_OK; ++i)
      st = launch_region<kWBf16>(c.plan[i], N, K, d_X, d_work, d_Y, y_bf16, stream, part);
  } else {
    for (int i = 0; i < c.count && st == Q4NX_OK; ++i)
      st = launch_region<WF>(c.plan[i], N, K, d_X, d_W, d_Y, y_bf16, stream, part);
  }
  if (st != Q4NX_OK) return st;
  return check_launch(fn);
}

static q4nx_status check_launch(const char* fn) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(Q4NX_ERR_HIP, std::string(fn) + ": " + hipGetErrorString(e));
  return Q4NX_OK;
}

// Row-group size: whole strips when there are enough of them to keep at least
// ~160 CUs streaming (one CU sustains ~55 GB/s of the ~7 TB/s), else halves or
// quarters of strips.  `strips` is the number of strips of the whole launch.
static int gemv_tq(int64_t strips) {
  if (strips >= 160) return 4;
  if (strips * 2 >= 160) return 2;
  return 1;
}

// Waves per workgroup (they split K).  A power of two, so that workgroups tile
// the 16 waves a CU holds at this kernel's register budget; fewer waves per
// row group when the launch has many row groups (longer streams per wave),
// more when it has few (more parallelism per strip).  Capped so every wave
// owns at least one block of every job.  Measured on MI355X over the Gemma3
// 1B/4B/27B projection shapes.
static int gemv_waves(int64_t row_groups, int min_kb) {
  int w = row_groups >= 4096 ? 2 : row_groups >= 512 ? 4 : row_groups >= 128 ? 8 : 16;
  while (w > 1 && w > min_kb) w >>= 1;
  return w;
}

template <int F>
static q4nx_status gemv_launch(const q4nx_gemv_desc* descs, int count, q4nx_dtype y_dtype, hipStream_t stream,
                               const char* fn) {
  clear_error();
  if (!descs || count < 1 || count > Q4NX_MAX_BATCH)
    return fail(Q4NX_ERR_INVALID_ARG, std::string(fn) + ": need 1..8 descriptors");
  if (y_dtype != Q4NX_F32 && y_dtype != Q4NX_BF16)
    return fail(Q4NX_ERR_INVALID_ARG, std::string(fn) + ": unknown y_dtype");
  int64_t strips = 0;
  for (int i = 0; i < count; ++i) {
    const q4nx_gemv_desc& d = descs[i];
    if (q4nx_status st = check_shape(d.N, d.K, fn)) return st;
    if (!d.blob || !d.x || !d.y) return fail(Q4NX_ERR_INVALID_ARG, std::string(fn) + ": NULL pointer");
    if (!aligned(d.blob, 16) || !aligned(d.x, 16) || !aligned(d.y, 4))
      return fail(Q4NX_ERR_ALIGNMENT, std::string(fn) + ": blob/x need 16-byte, y 4-byte alignment");
    strips += ceil_div(d.N, kBlockRows);
  }
  int min_kb = 1 << 30, max_kb = 0;
  for (int i = 0; i < count; ++i) {
    min_kb = std::min<int>(min_kb, (int)ceil_div(descs[i].K, kBlockCols));
    max_kb = std::max<int>(max_kb, (int)ceil_div(descs[i].K, kBlockCols));
  }
  // Launches of 80-159 strips take the streaming form with half-strip row
  // groups, 8 waves each.  Measured on MI355X in whole Gemma3 decode steps:
  // the 4B step 3% faster (its q/k/v, o and down launches); with quarter-strip
  // groups at 160-256 strips the 27B step was 2% slower (although each of
  // those launch types alone, repeated, ran 2-5% faster), so those launches
  // keep gemv_kernel.
  const bool streaming = max_kb <= kGemvChunkBlocks && strips >= 80 && strips < 160;
  const int tq = streaming ? 2 : gemv_tq(strips);
  int waves = streaming ? 8 : gemv_waves(strips * (4 / tq), min_kb);
  while (waves > 1 && waves > min_kb) waves >>= 1;
  GemvArgs args = {};
  args.njobs = count;
  args.y_bf16 = (y_dtype == Q4NX_BF16);
  int64_t wg = 0;
  int max_waves = 1;
  for (int i = 0; i < count; ++i) {
    const q4nx_gemv_desc& d = descs[i];
    GemvJob& J = args.job[i];
    J.blob = static_cast<const uint8_t*>(d.blob);
    J.x = d.x;
    J.y = d.y;
    J.N = (int)d.N;
    J.K = (int)d.K;
    J.NS = (int)ceil_div(d.N, kBlockRows);
    J.KB = (int)ceil_div(d.K, kBlockCols);
    J.tq = tq;
    J.nrg = J.NS * (4 / tq);
    J.waves = waves;
    // One workgroup per row group (the hardware keeps every CU fed as
    // workgroups retire); the loop over row groups only engages past 2^20.
    J.nwg = std::min(J.nrg, 1 << 20);
    J.wg_begin = (int)wg;
    wg += J.nwg;
    max_waves = std::max(max_waves, J.waves);
    args.chunk_blocks = std::max(args.chunk_blocks, std::min(J.KB, kGemvChunkBlocks));
  }
  // LDS of both kernels (static): the row sums and one x slot per wave.
  constexpr int64_t lds = sizeof(float) * (kRedFloats + kGemvMaxWaves * kGroupsPerRow * kGroupPadDw);
  const dim3 block(64 * max_waves);
  if (streaming) {
    // Streaming form: a bounded grid (workgroups per CU as the LDS allows, at
    // most kGemvStreamPerCu), dealt to the jobs in proportion to their row
    // groups; each workgroup walks its job's row groups r0, r0 + nwg, ...
    const int64_t per_cu = std::max<int64_t>(1, std::min<int64_t>(kGemvStreamPerCu, (160 * 1024) / lds));
    const int64_t total_rg = strips * (4 / tq), budget = (int64_t)device_cus() * per_cu;
    int64_t sw = 0;
    for (int i = 0; i < count; ++i) {
      GemvJob& J = args.job[i];
      J.nwg = (int)std::max<int64_t>(1, std::min<int64_t>(J.nrg, (budget * J.nrg + total_rg - 1) / total_rg));
      J.wg_begin = (int)sw;
      sw += J.nwg;
    }
    hipLaunchKernelGGL((gemv_stream_kernel<2, kGemvDepth2, F>), dim3((unsigned)sw), block, 0, stream, args);
    return check_launch(fn);
  }
  const dim3 grid((unsigned)wg);
  switch (tq) {  // x is staged per wave in static LDS
    case 4: hipLaunchKernelGGL((gemv_kernel<4, kGemvDepth4, F>), grid, block, 0, stream, args); break;
    case 2: hipLaunchKernelGGL((gemv_kernel<2, kGemvDepth2, F>), grid, block, 0, stream, args); break;
    default: hipLaunchKernelGGL((gemv_kernel<1, kGemvDepth1, F>), grid, block, 0, stream, args); break;
  }
  return check_launch(fn);
}

template <int F>
static q4nx_status dequant_entry(const void* d_blob, int64_t N, int64_t K, void* d_W, q4nx_dtype w_dtype,
                                 hipStream_t stream, const char* fn) {
  clear_error();
  if (q4nx_status st = check_shape(N, K, fn)) return st;
  if (!d_blob || !d_W) return fail(Q4NX_ERR_INVALID_ARG, std::string(fn) + ": NULL pointer");
  if (w_dtype != Q4NX_F32 && w_dtype != Q4NX_BF16)
    return fail(Q4NX_ERR_INVALID_ARG, std::string(fn) + ": unknown w_dtype");
  if (!aligned(d_blob, 16) || !aligned(d_W, 16))
    return fail(Q4NX_ERR_ALIGNMENT, std::string(fn) + ": blob and W need 16-byte alignment");
  const int64_t KB = ceil_div(K, kBlockCols);
  const int64_t nblocks = ceil_div(N, kBlockRows) * KB;
  const int64_t grid = std::min<int64_t>(nblocks, int64_t(1) << 20);
  const uint8_t* blob = static_cast<const uint8_t*>(d_blob);
  const int w_bf16 = (w_dtype == Q4NX_BF16);
  hipLaunchKernelGGL(dequant_kernel<F>, dim3((unsigned)grid), dim3(256), 0, stream, blob, N, K, KB, nblocks, d_W,
                     w_bf16);
  return check_launch(fn);
}

// Measurement aid: read a buffer once with the GEMV's load pattern (16-byte
// non-temporal loads, a workgroup per contiguous slice, through a buffer
// descriptor limited to the slice, so no load needs a bounds test) and fold it
// into one value per wave (lane shuffles, no LDS and no barrier), so that
// nothing is dead code and the kernel has no tail beyond the loads.  Gives the
// read bandwidth, and the per-launch floor, of a plain streaming kernel.
constexpr int kStreamWgs = 2048;
__global__ __launch_bounds__(256) void stream_read_kernel(const uint8_t* __restrict__ src, int64_t n16,
                                                          float* __restrict__ sink) {
  const int64_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const int64_t b = (int64_t)blockIdx.x * per, e = min(n16, b + per);
  const int cnt = (int)max<int64_t>(0, e - b);  // 16-byte pieces of this slice
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(src) + (e > b ? b * 16 : 0), (short)0, cnt * 16, 0x00020000);
  uint32_t acc = 0;
  for (int i = threadIdx.x; i < cnt; i += 4 * 256) {
    u32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      v[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (i + u * 256) * 16, 0, kNtLoad));
#pragma unroll
    for (int u = 0; u < 4; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  acc ^= (uint32_t)xor_lane_bits<32>((int)acc);
  acc ^= (uint32_t)xor_lane_bits<16>((int)acc);
  acc ^= (uint32_t)xor_lane_bits<8>((int)acc);
  acc ^= (uint32_t)xor_lane_bits<4>((int)acc);
  acc ^= (uint32_t)xor_lane_bits<2>((int)acc);
  acc ^= (uint32_t)xor_lane_bits<1>((int)acc);
  if ((threadIdx.x & 63) == 0) sink[blockIdx.x * 4 + (threadIdx.x >> 6)] = __uint_as_float(acc & 0x3FFFFFFFu);
}

}  // namespace q4nx

using namespace q4nx;

extern "C" {

q4nx_status q4nx_dequant(const void* d_blob, int64_t N, int64_t K, void* d_W, q4nx_dtype w_dtype,
                         hipStream_t stream) {
  return dequant_entry<kWQ4NX>(d_blob, N, K, d_W, w_dtype, stream, "q4nx_dequant");
}

q4nx_status q4nx_mx_dequant(const void* d_blob, int64_t N, int64_t K, void* d_W, q4nx_dtype w_dtype,
                            hipStream_t stream) {
  return dequant_entry<kWMX>(d_blob, N, K, d_W, w_dtype, stream, "q4nx_mx_dequant");
}

q4nx_status q4nx_quantize(const float* d_W, int64_t N, int64_t K, void* d_blob, hipStream_t stream) {
  clear_error();
  if (q4nx_status st = check_shape(N, K, "q4nx_quantize")) return st;
  if (!d_W || !d_blob) return fail(Q4NX_ERR_INVALID_ARG, "q4nx_quantize: NULL pointer");
  if (!aligned(d_W, 16) || !aligned(d_blob, 16))
    return fail(Q4NX_ERR_ALIGNMENT, "q4nx_quantize: W and blob need 16-byte alignment");
  const int64_t KB = ceil_div(K, kBlockCols);
  const int64_t nblocks = ceil_div(N, kBlockRows) * KB;
  const int64_t grid = std::min<int64_t>(nblocks, int64_t(1) << 20);
  hipLaunchKernelGGL(quantize_kernel, dim3((unsigned)grid), dim3(256), 0, stream, d_W, N, K, KB, nblocks,
                     static_cast<uint8_t*>(d_blob));
  return check_launch("q4nx_quantize");
}

q4nx_status q4nx_mx_quantize(const float* d_W, int64_t N, int64_t K, void* d_blob, hipStream_t stream) {
  clear_error();
  if (q4nx_status st = check_shape(N, K, "q4nx_mx_quantize")) return st;
  if (!d_W || !d_blob) return fail(Q4NX_ERR_INVALID_ARG, "q4nx_mx_quantize: NULL pointer");
  if (!aligned(d_W, 16) || !aligned(d_blob, 16))
    return fail(Q4NX_ERR_ALIGNMENT, "q4nx_mx_quantize: W and blob need 16-byte alignment");
  const int64_t KB = ceil_div(K, kBlockCols);
  const int64_t nblocks = ceil_div(N, kBlockRows) * KB;
  const int64_t grid = std::min<int64_t>(nblocks, int64_t(1) << 20);
  hipLaunchKernelGGL(mx_quantize_kernel, dim3((unsigned)grid), dim3(256), 0, stream, d_W, N, K, KB, nblocks,
                     static_cast<uint8_t*>(d_blob));
  return check_launch("q4nx_mx_quantize");
}

q4nx_status q4nx_stream_read(const void* d_src, size_t bytes, float* d_sink, hipStream_t stream) {
  clear_error();
  if (!d_src || !d_sink) return fail(Q4NX_ERR_INVALID_ARG, "q4nx_stream_read: NULL pointer");
  if (bytes == 0 || bytes % 16 != 0 || bytes / kStreamWgs >= (size_t(1) << 31))
    return fail(Q4NX_ERR_SHAPE, "q4nx_stream_read: bytes must be a positive multiple of 16, below 2^42");
  if (!aligned(d_src, 16) || !aligned(d_sink, 4)) return fail(Q4NX_ERR_ALIGNMENT, "q4nx_stream_read: src needs 16-byte alignment");
  hipLaunchKernelGGL(stream_read_kernel, dim3(kStreamWgs), dim3(256), 0, stream, static_cast<const uint8_t*>(d_src),
                     (int64_t)(bytes / 16), d_sink);
  return check_launch("q4nx_stream_read");
}

q4nx_status q4nx_gemv(const void* d_blob, const uint16_t* d_x, void* d_y, q4nx_dtype y_dtype, int64_t N,
                      int64_t K, hipStream_t stream) {
  q4nx_gemv_desc d = {d_blob, d_x, d_y, N, K};
  return gemv_launch<kWQ4NX>(&d, 1, y_dtype, stream, "q4nx_gemv");
}

q4nx_status q4nx_gemv_batched(const q4nx_gemv_desc* descs, int32_t count, q4nx_dtype y_dtype,
                              hipStream_t stream) {
  return gemv_launch<kWQ4NX>(descs, count, y_dtype, stream, "q4nx_gemv_batched");
}

q4nx_status q4nx_mx_gemv(const void* d_blob, const uint16_t* d_x, void* d_y, q4nx_dtype y_dtype, int64_t N,
                         int64_t K, hipStream_t stream) {
  q4nx_gemv_desc d = {d_blob, d_x, d_y, N, K};
  return gemv_launch<kWMX>(&d, 1, y_dtype, stream, "q4nx_mx_gemv");
}

q4nx_status q4nx_mx_gemv_batched(const q4nx_gemv_desc* descs, int32_t count, q4nx_dtype y_dtype,
                                 hipStream_t stream) {
  return gemv_launch<kWMX>(descs, count, y_dtype, stream, "q4nx_mx_gemv_batched");
}

q4nx_status q4nx_gemm(int64_t M, int64_t N, int64_t K, const uint16_t* d_X, const void* d_blob, void* d_Y,
                      q4nx_dtype y_dtype, hipStream_t stream) {
  return gemm_entry<kWQ4NX>(M, N, K, d_X, d_blob, d_Y, y_dtype, nullptr, 0, stream, "q4nx_gemm");
}

q4nx_status q4nx_mx_gemm(int64_t M, int64_t N, int64_t K, const uint16_t* d_X, const void* d_blob, void* d_Y,
                         q4nx_dtype y_dtype, hipStream_t stream) {
  return gemm_entry<kWMX>(M, N, K, d_X, d_blob, d_Y, y_dtype, nullptr, 0, stream, "q4nx_mx_gemm");
}

q4nx_status q4nx_gemm_bf16(int64_t M, int64_t N, int64_t K, const uint16_t* d_X, const uint16_t* d_W, void* d_Y,
                           q4nx_dtype y_dtype, hipStream_t stream) {
  return gemm_entry<kWBf16>(M, N, K, d_X, d_W, d_Y, y_dtype, nullptr, 0, stream, "q4nx_gemm_bf16");
}

size_t q4nx_gemm_workspace_size(q4nx_weights w_format, int64_t M, int64_t N, int64_t K) {
  if (M <= 0 || N <= 0 || K <= 0 || K % kGroup != 0 || M > Q4NX_MAX_DIM || N > Q4NX_MAX_DIM || K > Q4NX_MAX_DIM ||
      M * N > (int64_t(1) << 40))
    return 0;
  int wf;
  switch (w_format) {
    case Q4NX_WEIGHTS_Q4NX: wf = kWQ4NX; break;
    case Q4NX_WEIGHTS_MXFP4: wf = kWMX; break;
    case Q4NX_WEIGHTS_BF16: wf = kWBf16; break;
    default: return 0;
  }
  const GemmChoice c = gemm_choose(wf, M, N, K, true);
  return c.w_bytes + c.part_bytes;
}

q4nx_status q4nx_gemm_ex(q4nx_weights w_format, int64_t M, int64_t N, int64_t K, const uint16_t* d_X,
                         const void* d_W, void* d_Y, q4nx_dtype y_dtype, void* d_work, size_t work_bytes,
                         hipStream_t stream) {
  switch (w_format) {
    case Q4NX_WEIGHTS_Q4NX:
      return gemm_entry<kWQ4NX>(M, N, K, d_X, d_W, d_Y, y_dtype, d_work, work_bytes, stream, "q4nx_gemm_ex");
    case Q4NX_WEIGHTS_MXFP4:
      return gemm_entry<kWMX>(M, N, K, d_X, d_W, d_Y, y_dtype, d_work, work_bytes, stream, "q4nx_gemm_ex");
    case Q4NX_WEIGHTS_BF16:
      return gemm_entry<kWBf16>(M, N, K, d_X, d_W, d_Y, y_dtype, d_work, work_bytes, stream, "q4nx_gemm_ex");
    default:
      clear_error();
      return fail(Q4NX_ERR_INVALID_ARG, "q4nx_gemm_ex: unknown w_format");
  }
}

}  // extern "C"
