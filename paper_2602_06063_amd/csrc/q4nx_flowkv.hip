// FlowKV decode attention for gfx950: the attention of one decode position
// over the KV cache (the causal-attention equation of the decoding section),
// computed with FlowKV's chunk sweep (Eq. 6-12 with a query chunk of 1), with
// its sliding-window variant.
//
// The sweep is split in two launches.  Phase 1 gives every (KV group, chunk of
// 16, 32, 64, 128, 256 or 512 positions) to one workgroup, which computes for the H/G query heads
// of the group the chunk's own running state: the max score m_c (Eq. 7), the
// denominator l_c = sum exp(s - m_c) (Eq. 8, 10) and the weighted values
// Y_c = sum exp(s - m_c) v (Eq. 11), into the caller's workspace.  Phase 2
// merges the chunks of each head with the correction factor of Eq. 9 taken
// relative to the largest chunk max, which is what the left-to-right
// recurrence reaches after the last chunk, then divides (Eq. 12).  Reading the cache is the whole cost: each K and V
// row is read once, by one workgroup, with full 128-byte rows per load.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <string>
#include <type_traits>

#include "q4nx_device.h"
#include "q4nx_internal.h"
#include "q4nx_xlane.h"

namespace q4nx {

typedef __bf16 bf16x2f __attribute__((ext_vector_type(2)));

constexpr int kMinChunk = 16;      // smallest chunk: sizes the workspace
constexpr int kFkvThreads = 256;   // 4 waves
constexpr int kMergeRegs = 8;      // chunks per slice the one-pass merge holds in registers

// a.lo * b.lo + a.hi * b.hi + c for two bf16 pairs (exact products, float32 sum).
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2f, a), __builtin_bit_cast(bf16x2f, b), c, false);
}

__device__ __forceinline__ float bf16lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16hi(uint32_t v) { return __uint_as_float(v & 0xFFFF0000u); }

// Wave-wide reductions in a fixed order (deterministic): exchanges with lane
// l ^ 32, then ^ 16, ..., ^ 1.
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, xor_lane<32>(v));
  v = fmaxf(v, xor_lane<16>(v));
  v = fmaxf(v, xor_lane<8>(v));
  v = fmaxf(v, xor_lane<4>(v));
  v = fmaxf(v, xor_lane<2>(v));
  return fmaxf(v, xor_lane<1>(v));
}
__device__ __forceinline__ float wave_sum(float v) {
  v += xor_lane<32>(v);
  v += xor_lane<16>(v);
  v += xor_lane<8>(v);
  v += xor_lane<4>(v);
  v += xor_lane<2>(v);
  return v + xor_lane<1>(v);
}

// Sum over the lanes l ^ m for m = R, 2R, ..., 32 (R a power of two, 8 to
// 32), in that order.
template <int R>
__device__ __forceinline__ float sum_lanes_from(float v) {
  if constexpr (R <= 8) v += xor_lane<8>(v);
  if constexpr (R <= 16) v += xor_lane<16>(v);
  return v + xor_lane<32>(v);
}

// Phase 1.  grid (chunks, G); CH cache positions per workgroup, D = head
// dimension, HG = query heads per group.  Partial of (head, chunk) at
// work[(head * nchunks + chunk) * (D + 4)]: m_c, l_c, -, -, Y_c[D].
template <int CH, int D, int HG, bool PRE>
__global__ __launch_bounds__(kFkvThreads) void flowkv_chunk_kernel(const uint16_t* __restrict__ q,
                                                                  const uint16_t* __restrict__ K,
                                                                  const uint16_t* __restrict__ V, int64_t L,
                                                                  int j0, int j1, float scale,
                                                                  float* __restrict__ work) {
  constexpr int kPart = D + 4;
  // K and V rows in flight per lane: 4 for 512-byte rows (d = 256), 2 for
  // 256-byte rows, where a deeper unroll measured slower.
  constexpr int kFkvUnroll = D >= 256 ? 4 : 2;
  constexpr int R = D / 8;        // lanes per V row (16 bytes each)
  constexpr int P = 64 / R;       // V rows per wave load
  __shared__ __attribute__((aligned(16))) uint32_t qs[HG][D / 2];   // query bf16 pairs
  __shared__ float fs[CH][HG];                                       // scores, then exp(s - m_c)
  __shared__ float red[4][HG];
  __shared__ __attribute__((aligned(16))) float ys[4][HG][D];        // per-wave partial Y

  const int c = blockIdx.x, g = blockIdx.y, nchunks = gridDim.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int k0 = j0 + c * CH, n = min(j1 - k0, CH);   // positions k0 .. k0+n-1
  const uint16_t* Kg = K + (size_t)g * L * D + (size_t)k0 * D;
  const uint16_t* Vg = V + (size_t)g * L * D + (size_t)k0 * D;

  // Lane roles: scores use 8 lanes per position (8 x 16 B = one 128-byte
  // piece of the row per load; lane u of the 8 takes dims 64i + 8u .. +7),
  // the weighted values R lanes per row (16 bytes, 8 dims, each).
  const int u = lane & 7, kw = lane >> 3;
  const int rs = lane / R, db = lane % R;
  // PRE: the whole chunk's K and V pieces of this lane are requested before
  // the query is staged, so the three round trips overlap (the chunk's rows
  // sit in registers: kSIt x D / 64 K pieces and CH / (4P) V pieces, rounded
  // up; pieces past the chunk are not loaded).
  constexpr int kSIt = (CH + 31) / 32;  // score passes of 32 positions (one, partly used, for CH = 16)
  constexpr int kQPer = (HG * D / 2 + kFkvThreads - 1) / kFkvThreads;
  constexpr int kKIt = PRE ? kSIt : 1, kKPc = PRE ? D / 64 : 1, kVIt = PRE ? (CH + 4 * P - 1) / (4 * P) : 1;
  uint4 kreg[kKIt][kKPc], vreg[kVIt];
  uint32_t qreg[kQPer];
  if constexpr (PRE) {
#pragma unroll
    for (int o = 0; o < kQPer; ++o) {
      const int e = tid + o * kFkvThreads;
      if (e < HG * D / 2) {
        const int h = e / (D / 2), p = e % (D / 2);
        qreg[o] = reinterpret_cast<const uint32_t*>(q + (size_t)(g * HG + h) * D)[p];
      }
    }
#pragma unroll
    for (int r = 0; r < kKIt; ++r) {
      const int pl = (r * 4 + wave) * 8 + kw;
#pragma unroll
      for (int i = 0; i < kKPc; ++i)
        kreg[r][i] = pl < n ? reinterpret_cast<const uint4*>(Kg + (size_t)pl * D)[8 * i + u] : uint4{0, 0, 0, 0};
    }
#pragma unroll
    for (int it = 0; it < kVIt; ++it) {
      const int pl = wave * P + rs + it * 4 * P;
      vreg[it] = pl < n ? reinterpret_cast<const uint4*>(Vg + (size_t)pl * D)[db] : uint4{0, 0, 0, 0};
    }
#pragma unroll
    for (int o = 0; o < kQPer; ++o) {
      const int e = tid + o * kFkvThreads;
      if (e < HG * D / 2) qs[e / (D / 2)][e % (D / 2)] = qreg[o];
    }
  } else {
    for (int e = tid; e < HG * D / 2; e += kFkvThreads) {
      const int h = e / (D / 2), p = e % (D / 2);
      qs[h][p] = reinterpret_cast<const uint32_t*>(q + (size_t)(g * HG + h) * D)[p];
    }
  }
  __syncthreads();

  // Scores (Eq. 6).  (With PRE, kSIt <= kFkvUnroll: the loop unrolls fully
  // and kreg is indexed by constants.)
  static_assert(!PRE || kSIt <= kFkvUnroll, "PRE needs the score loop fully unrolled");
#pragma unroll kFkvUnroll
  for (int r = 0; r < kSIt; ++r) {
    const int pl = (r * 4 + wave) * 8 + kw;
    float acc[HG];
#pragma unroll
    for (int h = 0; h < HG; ++h) acc[h] = 0.0f;
    if (pl < n) {
      const uint4* row = reinterpret_cast<const uint4*>(Kg + (size_t)pl * D);
#pragma unroll
      for (int i = 0; i < D / 64; ++i) {
        uint4 kv;
        if constexpr (PRE) kv = kreg[r][i];
        else kv = row[8 * i + u];
#pragma unroll
        for (int h = 0; h < HG; ++h) {
          const uint4 qv = *reinterpret_cast<const uint4*>(&qs[h][32 * i + 4 * u]);
          acc[h] = dot2(kv.x, qv.x, acc[h]);
          acc[h] = dot2(kv.y, qv.y, acc[h]);
          acc[h] = dot2(kv.z, qv.z, acc[h]);
          acc[h] = dot2(kv.w, qv.w, acc[h]);
        }
      }
    }
#pragma unroll
    for (int h = 0; h < HG; ++h) {
      float v = acc[h];
      v += xor_lane<1>(v);
      v += xor_lane<2>(v);
      v += xor_lane<4>(v);
      if (u == 0 && pl < CH) fs[pl][h] = pl < n ? v * scale : -INFINITY;
    }
  }
  __syncthreads();

  // Chunk max (Eq. 7), exponentials (Eq. 8) and their sum (Eq. 10);
  // thread tid owns positions tid, tid + 256, ... below CH.
  constexpr int kOwn = (CH + kFkvThreads - 1) / kFkvThreads;
  float m[HG], l[HG];
#pragma unroll
  for (int h = 0; h < HG; ++h) {
    float v = -INFINITY;
#pragma unroll
    for (int o = 0; o < kOwn; ++o)
      if (tid + o * kFkvThreads < CH) v = fmaxf(v, fs[tid + o * kFkvThreads][h]);
    v = wave_max(v);
    if (lane == 0) red[wave][h] = v;
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < HG; ++h) m[h] = fmaxf(fmaxf(red[0][h], red[1][h]), fmaxf(red[2][h], red[3][h]));
  __syncthreads();
#pragma unroll
  for (int h = 0; h < HG; ++h) {
    float f = 0.0f;
#pragma unroll
    for (int o = 0; o < kOwn; ++o) {
      const int p = tid + o * kFkvThreads;
      if (p < CH) {
        const float e = expf(fs[p][h] - m[h]);   // exp(-inf) = 0 past the range
        fs[p][h] = e;
        f += e;
      }
    }
    const float sm = wave_sum(f);
    if (lane == 0) red[wave][h] = sm;
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < HG; ++h) l[h] = (red[0][h] + red[1][h]) + (red[2][h] + red[3][h]);

  // Weighted values (Eq. 11): wave w takes rows w*P + rs, then every 4P rows.
  float y[HG][8];
#pragma unroll
  for (int h = 0; h < HG; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) y[h][e] = 0.0f;
  // One V row piece (8 dims) of position pl into the weighted sums.
  const auto vrow = [&](int pl, const uint4 w) __attribute__((always_inline)) {
    const float v[8] = {bf16lo(w.x), bf16hi(w.x), bf16lo(w.y), bf16hi(w.y),
                        bf16lo(w.z), bf16hi(w.z), bf16lo(w.w), bf16hi(w.w)};
#pragma unroll
    for (int h = 0; h < HG; ++h) {
      const float f = fs[pl][h];
#pragma unroll
      for (int e = 0; e < 8; ++e) y[h][e] = fmaf(f, v[e], y[h][e]);
    }
  };
  if constexpr (PRE) {
#pragma unroll
    for (int it = 0; it < kVIt; ++it) {
      const int pl = wave * P + rs + it * 4 * P;
      if (pl < n) vrow(pl, vreg[it]);
    }
  } else {
#pragma unroll kFkvUnroll
    for (int pl = wave * P + rs; pl < n; pl += 4 * P) vrow(pl, reinterpret_cast<const uint4*>(Vg + (size_t)pl * D)[db]);
  }
  // Sum the P row slots of the wave (lanes db, db + R, ...), then the 4 waves.
#pragma unroll
  for (int h = 0; h < HG; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float v = y[h][e];
      v = sum_lanes_from<R>(v);
      y[h][e] = v;
    }
  if (rs == 0) {
#pragma unroll
    for (int h = 0; h < HG; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) ys[wave][h][8 * db + e] = y[h][e];
  }
  __syncthreads();

  for (int e = tid; e < HG * D; e += kFkvThreads) {
    const int h = e / D, dd = e % D;
    float* part = work + ((size_t)(g * HG + h) * nchunks + c) * kPart;
    part[4 + dd] = (ys[0][h][dd] + ys[1][h][dd]) + (ys[2][h][dd] + ys[3][h][dd]);
    if (dd == 0) {
      part[0] = m[h];
      part[1] = l[h];
    }
  }
}

// Phase 2.  grid (H, D / DW), 256 threads: workgroup (h, b) produces dims
// b*DW .. b*DW + DW-1 of head h, with S = 256 / DW slices of DW threads; slice
// s takes chunks s, s + S, ...  With M the largest chunk max, Eq. 9's
// correction of chunk c relative to M is exp(m_c - M); the head's output is
// sum_c exp(m_c - M) Y_c / sum_c exp(m_c - M) l_c (Eq. 10-12), summed over
// the chunks in increasing order within a slice and then over the slices
// (every workgroup of a head forms the same denominator in the same order).
// Splitting the dims keeps many chunks from serialising on a few workgroups
// when there are few heads (Gemma3 1B: 4 heads, 512 chunks at 32K).
template <int D, int DW, bool REGS>
__global__ __launch_bounds__(kFkvThreads) void flowkv_merge_kernel(const float* __restrict__ work, int nchunks,
                                                                   void* __restrict__ out, int out_bf16) {
  constexpr int kPart = D + 4, S = kFkvThreads / DW;
  __shared__ float mx[kFkvThreads / 64];
  __shared__ float ls[S], yls[S][DW];
  const int h = blockIdx.x, tid = threadIdx.x, dd = tid % DW, sl = tid / DW;
  const int dim = blockIdx.y * DW + dd;
  const float* part = work + (size_t)h * nchunks * kPart;
  // REGS (at most kMergeRegs chunks per slice): each thread reads its chunks'
  // (m_c, l_c, Y_c[dim]) once, in one round trip, and the block max comes
  // from those; otherwise the max and the sums read the partials in two
  // passes.  Either way M is the same maximum and the sums run over the same
  // chunks in the same order, so the bits do not depend on the path.
  constexpr bool in_regs = REGS;
  float pm[kMergeRegs], pl[kMergeRegs], py[kMergeRegs];
  float mloc = -INFINITY;
  if (in_regs) {
#pragma unroll
    for (int k = 0; k < kMergeRegs; ++k) {
      const int c = sl + k * S;
      pm[k] = -INFINITY;
      pl[k] = py[k] = 0.0f;
      if (c < nchunks) {
        const float* pc = part + (size_t)c * kPart;
        pm[k] = pc[0];
        pl[k] = pc[1];
        py[k] = pc[4 + dim];
      }
    }
#pragma unroll
    for (int k = 0; k < kMergeRegs; ++k) mloc = fmaxf(mloc, pm[k]);
  } else {
    for (int c = tid; c < nchunks; c += kFkvThreads) mloc = fmaxf(mloc, part[(size_t)c * kPart]);
  }
  mloc = wave_max(mloc);
  if ((tid & 63) == 0) mx[tid >> 6] = mloc;
  __syncthreads();
  float M = mx[0];
#pragma unroll
  for (int w = 1; w < kFkvThreads / 64; ++w) M = fmaxf(M, mx[w]);
  float l = 0.0f, y = 0.0f;
  if (in_regs) {
#pragma unroll
    for (int k = 0; k < kMergeRegs; ++k)
      if (sl + k * S < nchunks) {
        const float a = expf(pm[k] - M);
        l = fmaf(a, pl[k], l);
        y = fmaf(a, py[k], y);
      }
  } else {
#pragma unroll 4
    for (int c = sl; c < nchunks; c += S) {
      const float* pc = part + (size_t)c * kPart;
      const float a = expf(pc[0] - M);
      l = fmaf(a, pc[1], l);
      y = fmaf(a, pc[4 + dim], y);
    }
  }
  yls[sl][dd] = y;
  if (dd == 0) ls[sl] = l;
  __syncthreads();
  if (sl == 0) {
    float yt = yls[0][dd], lt = ls[0];
#pragma unroll
    for (int s2 = 1; s2 < S; ++s2) {
      yt += yls[s2][dd];
      lt += ls[s2];
    }
    const float o = yt / lt;
    if (out_bf16) {
      bf16x2f p = __builtin_convertvector((float __attribute__((ext_vector_type(2)))){o, 0.0f}, bf16x2f);
      static_cast<uint16_t*>(out)[(size_t)h * D + dim] = (uint16_t)(__builtin_bit_cast(uint32_t, p) & 0xFFFFu);
    } else {
      static_cast<float*>(out)[(size_t)h * D + dim] = o;
    }
  }
}

template <int CH, int D, int HG>
static void launch_flowkv(const uint16_t* q, const uint16_t* K, const uint16_t* V, int64_t L, int G, int j0, int j1,
                          float scale, float* work, void* out, int out_bf16, hipStream_t stream) {
  const int nchunks = (int)ceil_div(j1 - j0, CH);
  // Short ranges (at most 4096 positions, so chunks of 64 positions or fewer:
  // the sliding-window layers), which are latency-bound, request each chunk's K
  // and V with the query when there are at least 64 workgroups.  Measured on
  // MI355X over the Gemma3 layer stacks at 32K, same bits: 27B (256
  // workgroups per windowed layer) 3% and 4B (64) 2% faster.  Not with fewer
  // workgroups (1B's windowed layers: the V requests then delay the scores on
  // each CU's own bandwidth) nor on long ranges (1B's global layers also take
  // 64-position chunks, 512 workgroups: 2-5% slower with the early requests).
  bool pre = false;
  if constexpr (CH <= 64) {
    pre = (int64_t)nchunks * G >= 64 && j1 - j0 <= 4096;
    if (pre)
      hipLaunchKernelGGL((flowkv_chunk_kernel<CH, D, HG, true>), dim3(nchunks, G), dim3(kFkvThreads), 0, stream, q,
                         K, V, L, j0, j1, scale, work);
  }
  if (!pre)
    hipLaunchKernelGGL((flowkv_chunk_kernel<CH, D, HG, false>), dim3(nchunks, G), dim3(kFkvThreads), 0, stream, q, K,
                       V, L, j0, j1, scale, work);
  // Dims per merge workgroup: halved (down to 16) until there are at least
  // 128 workgroups.
  const int H = G * HG;
  int dw = D;
  while (dw > 16 && H * (D / dw) < 128) dw >>= 1;
  const dim3 mg(H, D / dw);
  // The one-pass merge where a slice takes at most kMergeRegs chunks.
  // Measured on MI355X over the Gemma3 layer stacks at 32K (same bits): 27B
  // 1.020 -> 0.995 ms, 4B 0.444 -> 0.436, 1B 0.330 -> 0.326.  (Both forms in
  // one kernel behind a run-time branch made the 1B stack 10% slower, so the
  // form is a template parameter.)
  const int slices = kFkvThreads / dw;
  const bool regs = nchunks <= slices * kMergeRegs;
  const auto merge = [&](auto dwc) {
    constexpr int DW = decltype(dwc)::value;
    if (regs)
      hipLaunchKernelGGL((flowkv_merge_kernel<D, DW, true>), mg, dim3(kFkvThreads), 0, stream, work, nchunks, out,
                         out_bf16);
    else
      hipLaunchKernelGGL((flowkv_merge_kernel<D, DW, false>), mg, dim3(kFkvThreads), 0, stream, work, nchunks, out,
                         out_bf16);
  };
  switch (dw) {
    case 256: merge(std::integral_constant<int, (D >= 256 ? 256 : D)>{}); break;
    case 128: merge(std::integral_constant<int, (D >= 128 ? 128 : D)>{}); break;
    case 64: merge(std::integral_constant<int, 64>{}); break;
    case 32: merge(std::integral_constant<int, 32>{}); break;
    default: merge(std::integral_constant<int, 16>{}); break;
  }
}

// Chunk size: the largest of 512, 256, 128, 64 positions that still gives at
// least two workgroups per CU; 32 where 64 leaves CUs without a workgroup,
// and 16 where 32 still gives fewer than 64 workgroups.  (Measured on MI355X
// over the Gemma3 layer stacks at 32K, windowed layers: the 4B stack 0.407 ms
// at 64 positions (64 workgroups per layer), 0.376 at 32 (128), 0.378 at 16
// (256); the 1B stack 0.287 ms at 64 (16 workgroups), 0.277 at 32 (32),
// 0.255 at 16 (64); the 27B windowed layers, 256 workgroups at 64, went 3%
// slower at 32.)
static int flowkv_chunk(int64_t n, int G, int cus) {
  for (int ch = 512; ch > 64; ch >>= 1)
    if (ceil_div(n, ch) * G >= 2 * cus) return ch;
  if (ceil_div(n, 64) * G >= cus) return 64;
  return ceil_div(n, 32) * G >= 64 ? 32 : kMinChunk;
}

template <int D, int HG>
static void launch_chunked(const uint16_t* q, const uint16_t* K, const uint16_t* V, int64_t L, int G, int j0, int j1,
                           float scale, float* work, void* out, int out_bf16, hipStream_t stream, int cus) {
  switch (flowkv_chunk(j1 - j0, G, cus)) {
    case 512: launch_flowkv<512, D, HG>(q, K, V, L, G, j0, j1, scale, work, out, out_bf16, stream); break;
    case 256: launch_flowkv<256, D, HG>(q, K, V, L, G, j0, j1, scale, work, out, out_bf16, stream); break;
    case 128: launch_flowkv<128, D, HG>(q, K, V, L, G, j0, j1, scale, work, out, out_bf16, stream); break;
    case 64: launch_flowkv<64, D, HG>(q, K, V, L, G, j0, j1, scale, work, out, out_bf16, stream); break;
    case 32: launch_flowkv<32, D, HG>(q, K, V, L, G, j0, j1, scale, work, out, out_bf16, stream); break;
    default: launch_flowkv<16, D, HG>(q, K, V, L, G, j0, j1, scale, work, out, out_bf16, stream); break;
  }
}

template <int D>
static bool dispatch_hg(int hg, const uint16_t* q, const uint16_t* K, const uint16_t* V, int64_t L, int G, int j0,
                        int j1, float scale, float* work, void* out, int out_bf16, hipStream_t stream, int cus) {
  switch (hg) {
    case 1: launch_chunked<D, 1>(q, K, V, L, G, j0, j1, scale, work, out, out_bf16, stream, cus); return true;
    case 2: launch_chunked<D, 2>(q, K, V, L, G, j0, j1, scale, work, out, out_bf16, stream, cus); return true;
    case 4: launch_chunked<D, 4>(q, K, V, L, G, j0, j1, scale, work, out, out_bf16, stream, cus); return true;
    case 8: launch_chunked<D, 8>(q, K, V, L, G, j0, j1, scale, work, out, out_bf16, stream, cus); return true;
    default: return false;
  }
}

// ---- scratch of the entry point that allocates nothing ----------------------
// q4nx_flowkv_decode_static keeps the chunk partials in this array instead of
// a caller workspace.  Each device holds its own copy, at its own address,
// for the life of the process.  Host code never passes the array's name to a
// kernel (on the host it is only a stand-in for the symbol): the device
// address comes from hipGetSymbolAddress, taken once per device with that
// device current.
constexpr size_t kStaticScratchBytes = Q4NX_FLOWKV_STATIC_BYTES;
static __device__ __align__(256) float scratch[kStaticScratchBytes / sizeof(float)];

static q4nx_status static_scratch(float** out) {
  static std::once_flag once[kMaxDevices];
  static float* ptr[kMaxDevices] = {};
  static hipError_t err[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return fail(Q4NX_ERR_HIP, "q4nx_flowkv_decode_static: no current device");
  std::call_once(once[dev], [&] {
    void* p = nullptr;
    err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    ptr[dev] = static_cast<float*>(p);
  });
  if (err[dev] != hipSuccess || ptr[dev] == nullptr)
    return fail(Q4NX_ERR_HIP, std::string("q4nx_flowkv_decode_static: hipGetSymbolAddress: ") +
                                  hipGetErrorString(err[dev]));
  *out = ptr[dev];
  return Q4NX_OK;
}

// Validation and launch shared by both entry points.  Every argument is
// checked before any HIP call.  work == nullptr selects the static scratch,
// whose need is sized by the chunk length the launch will use; a caller
// workspace is sized by the smallest chunk (q4nx_flowkv_workspace_size, which
// callers use to allocate before the chunk length is known).
static q4nx_status flowkv_entry(const uint16_t* d_q, const uint16_t* d_k, const uint16_t* d_v, int64_t H, int64_t G,
                                int64_t d, int64_t L, int64_t t, int64_t window, float scale, void* d_o,
                                q4nx_dtype o_dtype, float* work, size_t work_bytes, hipStream_t stream,
                                const char* fn) {
  const std::string f(fn);
  if (!d_q || !d_k || !d_v || !d_o) return fail(Q4NX_ERR_INVALID_ARG, f + ": NULL pointer");
  if (o_dtype != Q4NX_F32 && o_dtype != Q4NX_BF16) return fail(Q4NX_ERR_INVALID_ARG, f + ": unknown o_dtype");
  if (!std::isfinite(scale)) return fail(Q4NX_ERR_INVALID_ARG, f + ": scale must be finite");
  if (H <= 0 || G <= 0 || H % G != 0 || G > 65535) return fail(Q4NX_ERR_SHAPE, f + ": H must be a positive multiple of G");
  const int64_t hg = H / G;
  if (hg != 1 && hg != 2 && hg != 4 && hg != 8) return fail(Q4NX_ERR_SHAPE, f + ": H/G must be 1, 2, 4 or 8");
  if (d != 64 && d != 128 && d != 256) return fail(Q4NX_ERR_SHAPE, f + ": d must be 64, 128 or 256");
  if (L <= 0 || L > (int64_t(1) << 30) || t < 0 || t >= L || window < 0)
    return fail(Q4NX_ERR_SHAPE, f + ": need 0 <= t < L <= 2^30 and window >= 0");
  if (!aligned(d_q, 16) || !aligned(d_k, 16) || !aligned(d_v, 16) || !aligned(d_o, 4))
    return fail(Q4NX_ERR_ALIGNMENT, f + ": q, K and V need 16-byte alignment, o 4-byte");
  const int64_t j1 = t + 1, j0 = window == 0 ? 0 : std::max<int64_t>(0, j1 - window);
  if (work && work_bytes < q4nx_flowkv_workspace_size(H, d, j1 - j0))
    return fail(Q4NX_ERR_BUFFER_TOO_SMALL, f + ": workspace smaller than q4nx_flowkv_workspace_size");
  const int cus = current_device_cus();
  if (!work) {
    const size_t need = (size_t)H * (size_t)ceil_div(j1 - j0, flowkv_chunk(j1 - j0, (int)G, cus)) *
                        (size_t)(d + 4) * sizeof(float);
    if (need > kStaticScratchBytes)
      return fail(Q4NX_ERR_BUFFER_TOO_SMALL, f + ": the chunk partials (" + std::to_string(need) +
                                                 " bytes) exceed the static scratch (" +
                                                 std::to_string(kStaticScratchBytes) + " bytes)");
    if (q4nx_status st = static_scratch(&work)) return st;
  }
  const int ob = o_dtype == Q4NX_BF16;
  bool ok = false;
  if (d == 64) ok = dispatch_hg<64>((int)hg, d_q, d_k, d_v, L, (int)G, (int)j0, (int)j1, scale, work, d_o, ob, stream, cus);
  if (d == 128) ok = dispatch_hg<128>((int)hg, d_q, d_k, d_v, L, (int)G, (int)j0, (int)j1, scale, work, d_o, ob, stream, cus);
  if (d == 256) ok = dispatch_hg<256>((int)hg, d_q, d_k, d_v, L, (int)G, (int)j0, (int)j1, scale, work, d_o, ob, stream, cus);
  if (!ok) return fail(Q4NX_ERR_SHAPE, f + ": unsupported shape");
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(Q4NX_ERR_HIP, f + ": " + hipGetErrorString(e));
  return Q4NX_OK;
}

}  // namespace q4nx

using namespace q4nx;

extern "C" {

size_t q4nx_flowkv_workspace_size(int64_t H, int64_t d, int64_t n_keys) {
  if (H <= 0 || d <= 0 || n_keys <= 0 || H > (1 << 16) || d > 4096 || n_keys > (int64_t(1) << 30)) return 0;
  return (size_t)H * (size_t)ceil_div(n_keys, kMinChunk) * (size_t)(d + 4) * sizeof(float);
}

q4nx_status q4nx_flowkv_decode(const uint16_t* d_q, const uint16_t* d_k, const uint16_t* d_v, int64_t H, int64_t G,
                               int64_t d, int64_t L, int64_t t, int64_t window, float scale, void* d_o,
                               q4nx_dtype o_dtype, void* d_work, size_t work_bytes, hipStream_t stream) {
  clear_error();
  if (!d_work) return fail(Q4NX_ERR_INVALID_ARG, "q4nx_flowkv_decode: NULL pointer");
  if (!aligned(d_work, 16)) return fail(Q4NX_ERR_ALIGNMENT, "q4nx_flowkv_decode: workspace needs 16-byte alignment");
  return flowkv_entry(d_q, d_k, d_v, H, G, d, L, t, window, scale, d_o, o_dtype, static_cast<float*>(d_work),
                      work_bytes, stream, "q4nx_flowkv_decode");
}

q4nx_status q4nx_flowkv_decode_static(const uint16_t* d_q, const uint16_t* d_k, const uint16_t* d_v, int64_t H,
                                      int64_t G, int64_t d, int64_t L, int64_t t, int64_t window, float scale,
                                      void* d_o, q4nx_dtype o_dtype, hipStream_t stream) {
  clear_error();
  return flowkv_entry(d_q, d_k, d_v, H, G, d, L, t, window, scale, d_o, o_dtype, nullptr, 0, stream,
                      "q4nx_flowkv_decode_static");
}

}  // extern "C"
