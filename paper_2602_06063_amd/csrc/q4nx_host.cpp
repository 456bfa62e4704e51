// Host half of libq4nx: packing into / unpacking from the Q4NX layout
// (Sec. 3.1.1; layout described in include/q4nx.h), argument validation and
// error reporting.  Nothing here touches the GPU.
#include <algorithm>
#include <atomic>
#include <cstring>
#include <string>
#include <thread>
#include <vector>

#include "q4nx_internal.h"

namespace q4nx {

static thread_local std::string g_last_error;

q4nx_status fail(q4nx_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

void clear_error() { g_last_error.clear(); }

q4nx_status check_shape(int64_t N, int64_t K, const char* fn) {
  if (N <= 0 || K <= 0 || N > Q4NX_MAX_DIM || K > Q4NX_MAX_DIM)
    return fail(Q4NX_ERR_SHAPE, std::string(fn) + ": N and K must lie in 1..2^30");
  if (K % kGroup != 0)
    return fail(Q4NX_ERR_SHAPE, std::string(fn) + ": K must be a multiple of 32");
  return Q4NX_OK;
}

// A scale or offset is accepted when it is +-0 or a finite bf16 with biased
// exponent in [27, 227], i.e. magnitude in [2^-100, 2^101).
static inline bool in_domain(uint16_t b) {
  const uint16_t mag = b & 0x7FFF;
  if (mag == 0) return true;
  const int e = mag >> 7;
  return e >= 27 && e <= 227;
}

// Runs fn(begin, end) over [0, n) split across up to 16 host threads.
template <class F>
static void parallel_for(int64_t n, int64_t min_chunk, F fn) {
  unsigned hw = std::thread::hardware_concurrency();
  int64_t nt = std::max<int64_t>(1, std::min<int64_t>({(int64_t)(hw ? hw : 1), 16, n / std::max<int64_t>(1, min_chunk)}));
  if (nt <= 1) {
    fn((int64_t)0, n);
    return;
  }
  std::vector<std::thread> th;
  const int64_t chunk = ceil_div(n, nt);
  for (int64_t t = 0; t < nt; ++t) {
    const int64_t b = t * chunk, e = std::min(n, b + chunk);
    if (b >= e) break;
    th.emplace_back([=] { fn(b, e); });
  }
  for (auto& x : th) x.join();
}

}  // namespace q4nx

using namespace q4nx;

extern "C" {

size_t q4nx_packed_size(int64_t N, int64_t K) {
  if (N <= 0 || K <= 0 || N > Q4NX_MAX_DIM || K > Q4NX_MAX_DIM || K % kGroup != 0) return 0;
  return (size_t)(ceil_div(N, kBlockRows) * ceil_div(K, kBlockCols)) * (size_t)kBlockBytes;
}

q4nx_status q4nx_pack(const uint8_t* codes, const uint16_t* scales, const uint16_t* offsets,
                      int64_t N, int64_t K, void* blob, size_t blob_bytes) {
  clear_error();
  if (q4nx_status st = check_shape(N, K, "q4nx_pack")) return st;
  if (!codes || !scales || !offsets || !blob)
    return fail(Q4NX_ERR_INVALID_ARG, "q4nx_pack: NULL pointer");
  const size_t need = q4nx_packed_size(N, K);
  if (blob_bytes < need)
    return fail(Q4NX_ERR_BUFFER_TOO_SMALL, "q4nx_pack: blob_bytes < q4nx_packed_size(N, K)");

  const int64_t G = K / kGroup;
  // Validate everything before writing anything.
  std::atomic<int64_t> bad_code{-1}, bad_val{-1};
  parallel_for(N, 64, [&](int64_t r0, int64_t r1) {
    for (int64_t r = r0; r < r1; ++r) {
      const uint8_t* c = codes + r * K;
      uint8_t acc = 0;
      for (int64_t k = 0; k < K; ++k) acc |= c[k];
      if (acc & 0xF0) {
        for (int64_t k = 0; k < K; ++k)
          if (c[k] > 15) { bad_code.store(r * K + k); break; }
      }
      for (int64_t g = 0; g < G; ++g) {
        if (!in_domain(scales[r * G + g]) || !in_domain(offsets[r * G + g])) {
          bad_val.store(r * G + g);
          break;
        }
      }
    }
  });
  if (bad_code.load() >= 0)
    return fail(Q4NX_ERR_INVALID_ARG, "q4nx_pack: code > 15 at flat index " + std::to_string(bad_code.load()));
  if (bad_val.load() >= 0)
    return fail(Q4NX_ERR_INVALID_ARG,
                "q4nx_pack: scale or offset outside {0} U [2^-100, 2^101) at group index " +
                    std::to_string(bad_val.load()));

  const int64_t NS = ceil_div(N, kBlockRows), KB = ceil_div(K, kBlockCols);
  uint8_t* out = static_cast<uint8_t*>(blob);
  parallel_for(NS, 4, [&](int64_t s0, int64_t s1) {
    for (int64_t i = s0; i < s1; ++i) {
      for (int64_t j = 0; j < KB; ++j) {
        uint8_t* blk = out + (i * KB + j) * kBlockBytes;
        std::memset(blk, 0, kBlockBytes);
        uint8_t* sc = blk + kCodeBytes;
        uint8_t* of = sc + kScaleBytes;
        for (int r = 0; r < kBlockRows; ++r) {
          const int64_t n = i * kBlockRows + r;
          if (n >= N) break;
          const int64_t k0 = j * kBlockCols;
          const int64_t kn = std::min<int64_t>(kBlockCols, K - k0);
          const uint8_t* src = codes + n * K + k0;
          uint8_t* dst = blk + r * (kBlockCols / 2);
          for (int64_t c = 0; c + 1 < kn; c += 2) dst[c / 2] = (uint8_t)(src[c] | (src[c + 1] << 4));
          for (int64_t g = 0; g < kn / kGroup; ++g) {
            const uint16_t s = scales[n * G + k0 / kGroup + g];
            const uint16_t o = offsets[n * G + k0 / kGroup + g];
            const int idx = r * kGroupsPerRow + (int)g;
            sc[2 * idx] = (uint8_t)(s & 0xFF);
            sc[2 * idx + 1] = (uint8_t)(s >> 8);
            of[2 * idx] = (uint8_t)(o & 0xFF);
            of[2 * idx + 1] = (uint8_t)(o >> 8);
          }
        }
      }
    }
  });
  return Q4NX_OK;
}

q4nx_status q4nx_unpack(const void* blob, size_t blob_bytes, int64_t N, int64_t K,
                        uint8_t* codes, uint16_t* scales, uint16_t* offsets) {
  clear_error();
  if (q4nx_status st = check_shape(N, K, "q4nx_unpack")) return st;
  if (!blob || !codes || !scales || !offsets)
    return fail(Q4NX_ERR_INVALID_ARG, "q4nx_unpack: NULL pointer");
  if (blob_bytes < q4nx_packed_size(N, K))
    return fail(Q4NX_ERR_BUFFER_TOO_SMALL, "q4nx_unpack: blob_bytes < q4nx_packed_size(N, K)");
  const int64_t G = K / kGroup, KB = ceil_div(K, kBlockCols);
  const uint8_t* in = static_cast<const uint8_t*>(blob);
  parallel_for(N, 64, [&](int64_t r0, int64_t r1) {
    for (int64_t n = r0; n < r1; ++n) {
      const int64_t i = n / kBlockRows, r = n % kBlockRows;
      for (int64_t k = 0; k < K; ++k) {
        const int64_t j = k / kBlockCols, c = k % kBlockCols;
        const uint8_t byte = in[(i * KB + j) * kBlockBytes + r * (kBlockCols / 2) + c / 2];
        codes[n * K + k] = (c & 1) ? (byte >> 4) : (byte & 0x0F);
      }
      for (int64_t g = 0; g < G; ++g) {
        const int64_t j = g / kGroupsPerRow, c = g % kGroupsPerRow;
        const uint8_t* blk = in + (i * KB + j) * kBlockBytes;
        const int64_t idx = r * kGroupsPerRow + c;
        scales[n * G + g] = (uint16_t)(blk[kCodeBytes + 2 * idx] | (blk[kCodeBytes + 2 * idx + 1] << 8));
        offsets[n * G + g] = (uint16_t)(blk[kCodeBytes + kScaleBytes + 2 * idx] |
                                        (blk[kCodeBytes + kScaleBytes + 2 * idx + 1] << 8));
      }
    }
  });
  return Q4NX_OK;
}

size_t q4nx_mx_packed_size(int64_t N, int64_t K) {
  if (N <= 0 || K <= 0 || K % kGroup != 0 || N > Q4NX_MAX_DIM || K > Q4NX_MAX_DIM) return 0;
  return (size_t)ceil_div(N, kBlockRows) * (size_t)ceil_div(K, kBlockCols) * (size_t)kMxBlockBytes;
}

q4nx_status q4nx_mx_pack(const uint8_t* codes, const uint8_t* scales, int64_t N, int64_t K, void* blob,
                         size_t blob_bytes) {
  clear_error();
  if (q4nx_status st = check_shape(N, K, "q4nx_mx_pack")) return st;
  if (!codes || !scales || !blob) return fail(Q4NX_ERR_INVALID_ARG, "q4nx_mx_pack: NULL pointer");
  if (blob_bytes < q4nx_mx_packed_size(N, K))
    return fail(Q4NX_ERR_BUFFER_TOO_SMALL, "q4nx_mx_pack: blob_bytes < q4nx_mx_packed_size(N, K)");
  const int64_t G = K / kGroup;
  // Validate everything before writing anything.
  std::atomic<int64_t> bad_code{-1}, bad_val{-1};
  parallel_for(N, 64, [&](int64_t r0, int64_t r1) {
    for (int64_t r = r0; r < r1; ++r) {
      const uint8_t* c = codes + r * K;
      uint8_t acc = 0;
      for (int64_t k = 0; k < K; ++k) acc |= c[k];
      if (acc & 0xF0) {
        for (int64_t k = 0; k < K; ++k)
          if (c[k] > 15) { bad_code.store(r * K + k); break; }
      }
      for (int64_t g = 0; g < G; ++g)
        if (scales[r * G + g] < kMxExpMin || scales[r * G + g] > kMxExpMax) {
          bad_val.store(r * G + g);
          break;
        }
    }
  });
  if (bad_code.load() >= 0)
    return fail(Q4NX_ERR_INVALID_ARG, "q4nx_mx_pack: code > 15 at flat index " + std::to_string(bad_code.load()));
  if (bad_val.load() >= 0)
    return fail(Q4NX_ERR_INVALID_ARG, "q4nx_mx_pack: E8M0 scale outside [27, 227] at group index " +
                                          std::to_string(bad_val.load()));
  const int64_t NS = ceil_div(N, kBlockRows), KB = ceil_div(K, kBlockCols);
  uint8_t* out = static_cast<uint8_t*>(blob);
  parallel_for(NS, 4, [&](int64_t s0, int64_t s1) {
    for (int64_t i = s0; i < s1; ++i) {
      for (int64_t j = 0; j < KB; ++j) {
        uint8_t* blk = out + (i * KB + j) * kMxBlockBytes;
        std::memset(blk, 0, kCodeBytes);
        std::memset(blk + kCodeBytes, kMxPadScale, kMxScaleBytes);
        for (int r = 0; r < kBlockRows; ++r) {
          const int64_t n = i * kBlockRows + r;
          if (n >= N) break;
          const int64_t k0 = j * kBlockCols;
          const int64_t kn = std::min<int64_t>(kBlockCols, K - k0);
          const uint8_t* src = codes + n * K + k0;
          uint8_t* dst = blk + r * (kBlockCols / 2);
          for (int64_t c = 0; c + 1 < kn; c += 2) dst[c / 2] = (uint8_t)(src[c] | (src[c + 1] << 4));
          for (int64_t g = 0; g < kn / kGroup; ++g)
            blk[kCodeBytes + r * kGroupsPerRow + g] = scales[n * G + k0 / kGroup + g];
        }
      }
    }
  });
  return Q4NX_OK;
}

q4nx_status q4nx_mx_unpack(const void* blob, size_t blob_bytes, int64_t N, int64_t K, uint8_t* codes,
                           uint8_t* scales) {
  clear_error();
  if (q4nx_status st = check_shape(N, K, "q4nx_mx_unpack")) return st;
  if (!blob || !codes || !scales) return fail(Q4NX_ERR_INVALID_ARG, "q4nx_mx_unpack: NULL pointer");
  if (blob_bytes < q4nx_mx_packed_size(N, K))
    return fail(Q4NX_ERR_BUFFER_TOO_SMALL, "q4nx_mx_unpack: blob_bytes < q4nx_mx_packed_size(N, K)");
  const int64_t G = K / kGroup, KB = ceil_div(K, kBlockCols);
  const uint8_t* in = static_cast<const uint8_t*>(blob);
  parallel_for(N, 64, [&](int64_t r0, int64_t r1) {
    for (int64_t n = r0; n < r1; ++n) {
      const int64_t i = n / kBlockRows, r = n % kBlockRows;
      for (int64_t k = 0; k < K; ++k) {
        const uint8_t* blk = in + (i * KB + k / kBlockCols) * kMxBlockBytes;
        const uint8_t b = blk[r * (kBlockCols / 2) + (k % kBlockCols) / 2];
        codes[n * K + k] = (k & 1) ? (b >> 4) : (b & 0xF);
      }
      for (int64_t g = 0; g < G; ++g) {
        const uint8_t* blk = in + (i * KB + (g * kGroup) / kBlockCols) * kMxBlockBytes;
        scales[n * G + g] = blk[kCodeBytes + r * kGroupsPerRow + g % kGroupsPerRow];
      }
    }
  });
  return Q4NX_OK;
}

const char* q4nx_status_str(q4nx_status s) {
  switch (s) {
    case Q4NX_OK: return "ok";
    case Q4NX_ERR_INVALID_ARG: return "invalid argument";
    case Q4NX_ERR_SHAPE: return "invalid shape";
    case Q4NX_ERR_ALIGNMENT: return "misaligned pointer";
    case Q4NX_ERR_BUFFER_TOO_SMALL: return "buffer too small";
    case Q4NX_ERR_HIP: return "HIP error";
    default: break;
  }
  return "unknown status";
}

const char* q4nx_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
