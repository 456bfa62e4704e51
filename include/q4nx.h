/*
 * q4nx.h -- C ABI of libq4nx.so: the Q4NX 4-bit weight format and its
 * dequantization fused with the linear projection, for AMD Instinct MI355X
 * (gfx950).
 *
 * The format and the operations follow "Mapping Gemma3 onto an Edge Dataflow
 * Architecture" (arXiv 2602.06063):
 *   - Q4NX block (Sec. 3.1.1, Dequantization Engine): 32 x 256 int4 weights,
 *     256 bf16 scales and 256 bf16 minimal-value offsets, 5120 bytes; one
 *     scale/offset pair per group of 32 weights.
 *   - Dequantization, Eq. 3: w = d_g * q + m_g, q in {0..15}.
 *   - Decode projection (FusedDQP, Sec. 3.2.1, Eq. 14/15): y = W x with the
 *     dequantization fused into the mat-vec.
 *   - Prefill projection (Sec. 3.1.2): the tiled matrix product C = A x B,
 *     here Y = X W^T with W dequantized to bf16 on the fly.
 *
 * Conventions used by every function:
 *   - Shapes: M = token rows, N = output features, K = input features.  The
 *     weight matrix W is N x K.  K must be a multiple of 32 (the group size).
 *   - bf16 values travel as raw uint16_t bit patterns.
 *   - Layout of a packed matrix ("blob"): ceil(N/32) * ceil(K/256) blocks of
 *     5120 bytes, strip-major: block (i, j) -- rows 32i..32i+31, columns
 *     256j..256j+255 -- starts at byte (i * ceil(K/256) + j) * 5120.  Inside a
 *     block: 4096 bytes of codes (row r at byte 128r; byte c of a row holds
 *     column 2c in bits 0-3 and column 2c+1 in bits 4-7), then 256 scales,
 *     then 256 offsets, each indexed 8r + g for group g (columns 32g..32g+31)
 *     of row r, little-endian bf16.  Rows >= N and columns >= K are padding
 *     with code 0, scale +0 and offset +0.
 *   - Value domain of scales and offsets: zero, or a finite bf16 whose
 *     magnitude lies in [2^-100, 2^101).  Inside it Eq. 3 is exact up to one
 *     rounding in float32 and never produces a subnormal, so results do not
 *     depend on denormal flushing or on FMA contraction.
 *   - Ownership: the caller owns every buffer; the library never frees or
 *     retains caller memory.  Device pointers come from hipMalloc (or a
 *     framework allocator built on it).
 *   - Device calls validate their arguments synchronously on the host, before
 *     any HIP call, then only enqueue work on `stream` (NULL = the default
 *     stream) and return; they never synchronize the device.  A launch failure
 *     is reported as Q4NX_ERR_HIP (details in q4nx_last_error()).
 *   - The library allocates no device memory of its own: every kernel works
 *     in the caller's buffers plus on-chip memory, so calls may be captured
 *     in HIP graphs and may run concurrently on different streams (as long as
 *     their output buffers do not overlap).
 *   - No C++ exception crosses this interface.
 */
#ifndef Q4NX_H
#define Q4NX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

struct ihipStream_t;
typedef struct ihipStream_t* hipStream_t;

/* The two range enumerators of the enums passed into the library make every
 * 32-bit int a value of the type, so that an unknown value from a caller is
 * well defined and rejected (Q4NX_ERR_INVALID_ARG, or "unknown status") (without them only the
 * named values are valid values of the type in C++). */
typedef enum q4nx_status {
  Q4NX_OK = 0,
  Q4NX_ERR_INVALID_ARG = 1,      /* NULL pointer, unknown dtype, code > 15, scale/offset outside the domain */
  Q4NX_ERR_SHAPE = 2,            /* M, N or K <= 0, K % 32 != 0, or a size beyond the supported range */
  Q4NX_ERR_ALIGNMENT = 3,        /* device pointer not aligned as documented */
  Q4NX_ERR_BUFFER_TOO_SMALL = 4, /* blob_bytes < q4nx_packed_size(N, K) */
  Q4NX_ERR_HIP = 5,              /* a HIP runtime call or kernel launch failed */
  Q4NX_STATUS_RANGE_MIN_ = -2147483647 - 1,
  Q4NX_STATUS_RANGE_MAX_ = 2147483647
} q4nx_status;

typedef enum q4nx_dtype {
  Q4NX_F32 = 0,  /* float32 */
  Q4NX_BF16 = 1, /* bfloat16, round to nearest even from the float32 value */
  Q4NX_DTYPE_RANGE_MIN_ = -2147483647 - 1,
  Q4NX_DTYPE_RANGE_MAX_ = 2147483647
} q4nx_dtype;

/* Largest N and K accepted by every call (both < 2^31). */
#define Q4NX_MAX_DIM ((int64_t)1 << 30)

/*
 * Bytes of a packed N x K matrix: ceil(N/32) * ceil(K/256) * 5120 (Sec. 3.1.1:
 * 5120 bytes per 32 x 256 block).  Returns 0 if N <= 0, K <= 0, K % 32 != 0
 * or either exceeds Q4NX_MAX_DIM.
 */
size_t q4nx_packed_size(int64_t N, int64_t K);

/*
 * Host, synchronous.  Packs a quantized matrix into the Q4NX layout above --
 * the offline conversion of Sec. 3.1.1 (offsets pre-converted to bf16).
 *   codes   : N*K bytes, row-major [N][K], each 0..15 (q of Eq. 3)
 *   scales  : N*(K/32) bf16 bit patterns, row-major [N][K/32] (d_g of Eq. 3)
 *   offsets : N*(K/32) bf16 bit patterns, row-major [N][K/32] (m_g of Eq. 3)
 *   blob    : host buffer of blob_bytes >= q4nx_packed_size(N, K); all of
 *             its first q4nx_packed_size(N, K) bytes are written (padding 0).
 * Errors: Q4NX_ERR_INVALID_ARG (NULL pointer, code > 15, scale or offset
 * outside the value domain -- checked before anything is written),
 * Q4NX_ERR_SHAPE, Q4NX_ERR_BUFFER_TOO_SMALL.  Uses several host threads.
 */
q4nx_status q4nx_pack(const uint8_t* codes, const uint16_t* scales, const uint16_t* offsets,
                      int64_t N, int64_t K, void* blob, size_t blob_bytes);

/*
 * Host, synchronous.  The inverse of q4nx_pack (a test and inspection aid):
 * reads blob (blob_bytes >= q4nx_packed_size(N, K)) and writes codes [N][K],
 * scales [N][K/32] and offsets [N][K/32].  Errors: Q4NX_ERR_INVALID_ARG,
 * Q4NX_ERR_SHAPE, Q4NX_ERR_BUFFER_TOO_SMALL.
 */
q4nx_status q4nx_unpack(const void* blob, size_t blob_bytes, int64_t N, int64_t K,
                        uint8_t* codes, uint16_t* scales, uint16_t* offsets);

/*
 * Device.  The dequantization engine of Sec. 3.1.1: writes every weight of
 * the packed matrix, dequantized with Eq. 3, to d_W (row-major [N][K]).
 *   d_blob  : device, q4nx_packed_size(N, K) bytes, 16-byte aligned
 *   d_W     : device, N*K elements of w_dtype, 16-byte aligned
 *   w_dtype : Q4NX_F32 -> RN_fp32(d*q + m) exactly;
 *             Q4NX_BF16 -> that value rounded to bf16 (nearest even)
 * Errors: Q4NX_ERR_INVALID_ARG, Q4NX_ERR_SHAPE, Q4NX_ERR_ALIGNMENT, Q4NX_ERR_HIP.
 */
q4nx_status q4nx_dequant(const void* d_blob, int64_t N, int64_t K,
                         void* d_W, q4nx_dtype w_dtype, hipStream_t stream);

/*
 * Device.  Quantizer into Q4NX: the offline conversion of float32 weights into
 * the packed format that the paper performs before inference (Sec. 3.1.1:
 * per-group scale and minimal-value offset, groups of 32 as in Q4_1), written
 * straight into a blob.  Per group of 32 consecutive input columns:
 *   w -> 0 if NaN, else clamped to [-2^100, 2^100];
 *   lo, hi = min and max of the group (a zero minimum is +0);
 *   d = RNE_bf16(RN_fp32(RN_fp32(hi - lo) / 15)), m = RNE_bf16(lo), each
 *   flushed to a signed zero if its magnitude is below 2^-100;
 *   q = the code 0..15 whose Eq. 3 value RN_fp32(d*q + m) is nearest to w
 *   (differences taken in float64), the smaller code on a tie.
 *   d_W    : device, row-major [N][K] float32, 16-byte aligned
 *   d_blob : device, q4nx_packed_size(N, K) bytes, 16-byte aligned; fully
 *            written, padding included (code 0, scale +0, offset +0)
 * Every input value is accepted (the clamp above), so no device-side error
 * exists.  Errors: Q4NX_ERR_INVALID_ARG, Q4NX_ERR_SHAPE, Q4NX_ERR_ALIGNMENT,
 * Q4NX_ERR_HIP.
 */
q4nx_status q4nx_quantize(const float* d_W, int64_t N, int64_t K, void* d_blob, hipStream_t stream);

/*
 * Device.  FusedDQP (Sec. 3.2.1, Eq. 14/15): y[n] = sum_k w[n][k] * x[k] with
 * w from Eq. 3, dequantized in registers and never written to memory; float32
 * accumulation.
 *   d_blob : device, packed N x K matrix, 16-byte aligned
 *   d_x    : device, K bf16 values, 16-byte aligned
 *   d_y    : device, N values of y_dtype, 4-byte aligned; fully overwritten
 *            (no zeroing needed); nothing beyond N is written
 * Deterministic: the same call gives the same bits every time.
 * Errors: Q4NX_ERR_INVALID_ARG, Q4NX_ERR_SHAPE, Q4NX_ERR_ALIGNMENT, Q4NX_ERR_HIP.
 */
q4nx_status q4nx_gemv(const void* d_blob, const uint16_t* d_x, void* d_y, q4nx_dtype y_dtype,
                      int64_t N, int64_t K, hipStream_t stream);

/*
 * One independent projection for q4nx_gemv_batched: y = W x as in q4nx_gemv.
 */
typedef struct q4nx_gemv_desc {
  const void* blob;   /* device, packed N x K matrix, 16-byte aligned */
  const uint16_t* x;  /* device, K bf16 values, 16-byte aligned */
  void* y;            /* device, N outputs of the batch's y_dtype, 4-byte aligned */
  int64_t N;
  int64_t K;
} q4nx_gemv_desc;

#define Q4NX_MAX_BATCH 8

/*
 * Device.  Runs 1..Q4NX_MAX_BATCH independent FusedDQP projections in one
 * launch -- e.g. the q/k/v projections of a layer, or gate/up, which read the
 * same activation.  Each result meets the same error bound as q4nx_gemv (the
 * work split, hence the float32 summation order, is chosen for the launch as
 * a whole); repeating a call with the same descriptors reproduces it bit for
 * bit.  Outputs must not overlap inputs or each other.
 * Errors: as q4nx_gemv, for any descriptor; Q4NX_ERR_INVALID_ARG for a
 * count outside 1..Q4NX_MAX_BATCH.
 */
q4nx_status q4nx_gemv_batched(const q4nx_gemv_desc* descs, int32_t count, q4nx_dtype y_dtype,
                              hipStream_t stream);

/*
 * Device.  Prefill projection (Sec. 3.1.2, C = A x B with A = X, B = W^T):
 * Y[m][n] = sum_k X[m][k] * w[n][k], where each weight is dequantized with
 * Eq. 3 and rounded to bf16 (the paper dequantizes to bf16 before its MM),
 * the products are bf16 x bf16 on the matrix cores and the sums are float32.
 *   d_X : device, row-major [M][K] bf16, 16-byte aligned, K*2 % 16 == 0
 *         holds because K % 32 == 0
 *   d_blob : device, packed N x K matrix, 16-byte aligned
 *   d_Y : device, row-major [M][N] of y_dtype, 16-byte aligned; fully
 *         overwritten, nothing outside [M][N] is written
 * Errors: Q4NX_ERR_INVALID_ARG, Q4NX_ERR_SHAPE, Q4NX_ERR_ALIGNMENT, Q4NX_ERR_HIP.
 */
q4nx_status q4nx_gemm(int64_t M, int64_t N, int64_t K, const uint16_t* d_X, const void* d_blob,
                      void* d_Y, q4nx_dtype y_dtype, hipStream_t stream);

/*
 * Device.  Plain bf16 matrix product Y[m][n] = sum_k X[m][k] * W[n][k] with W
 * given in bf16 -- the second phase of the paper's two-phase prefill, where
 * the dequantization engine writes the bf16 weights that the MM then consumes
 * (Sec. 3.1.1 and 3.1.2): q4nx_dequant(blob, Q4NX_BF16) followed by this call.
 * The arithmetic is that of q4nx_gemm (bf16 x bf16 products on the matrix
 * cores, float32 sums over K in increasing order), so with W from
 * q4nx_dequant the result equals q4nx_gemm on the packed matrix bit for bit.
 *   d_X : device, row-major [M][K] bf16, 16-byte aligned
 *   d_W : device, row-major [N][K] bf16, 16-byte aligned (the caller owns it)
 *   d_Y : device, row-major [M][N] of y_dtype, 16-byte aligned; fully
 *         overwritten, nothing outside [M][N] is written
 * K must be a multiple of 32, as for q4nx_gemm.
 * Errors: Q4NX_ERR_INVALID_ARG, Q4NX_ERR_SHAPE, Q4NX_ERR_ALIGNMENT, Q4NX_ERR_HIP.
 */
q4nx_status q4nx_gemm_bf16(int64_t M, int64_t N, int64_t K, const uint16_t* d_X, const uint16_t* d_W,
                           void* d_Y, q4nx_dtype y_dtype, hipStream_t stream);

/* Smallest chunk (cache positions per workgroup) of q4nx_flowkv_decode. */
#define Q4NX_FLOWKV_MIN_CHUNK 16

/*
 * Bytes of the workspace q4nx_flowkv_decode needs for H query heads of
 * dimension d attending to n_keys cache positions:
 * H * ceil(n_keys / 16) * (d + 4) * 4.  Returns 0 for a non-positive or
 * out-of-range argument.
 */
size_t q4nx_flowkv_workspace_size(int64_t H, int64_t d, int64_t n_keys);

/*
 * Device.  FlowKV decode attention (Sec. 3.2.2, FlowKV and FlowKV-SWA): the
 * attention output of decode position t over the KV cache of positions
 * 0..t (the causal-attention equation of Sec. 2.2, with the score scaling of
 * Eq. 6 passed as `scale`, 1/sqrt(d) in the paper), computed with FlowKV's
 * chunk sweep (Eq. 6-12 with a query chunk of 1):
 *   o[h] = sum_j softmax_j(scale * q[h] . k[g][j]) v[g][j],  g = h / (H/G),
 *   j over 0..t (window == 0) or max(0, t-window+1)..t (window > 0, SWA).
 *   d_q     : device, [H][d] bf16, 16-byte aligned
 *   d_k,d_v : device, [G][L][d] bf16 (row j of group g = cache position j);
 *             only positions of the attended range are read; 16-byte aligned
 *   H, G    : query heads and KV groups (GQA), H/G in {1, 2, 4, 8}
 *   d       : head dimension, 64, 128 or 256
 *   L       : cache capacity (row count per group), 0 <= t < L <= 2^30
 *   d_o     : device, [H][d] of o_dtype, 4-byte aligned; fully written
 *   d_work  : device, >= q4nx_flowkv_workspace_size(H, d, attended length)
 *             bytes, 16-byte aligned, owned by the caller; its contents on
 *             entry do not matter and are overwritten
 * Scores are float32 sums of exact bf16 products; exponentials, sums and
 * the final division are float32.  Calls that share a workspace must not
 * overlap.  Errors: Q4NX_ERR_INVALID_ARG (NULL pointer, unknown dtype,
 * non-finite scale), Q4NX_ERR_SHAPE, Q4NX_ERR_ALIGNMENT,
 * Q4NX_ERR_BUFFER_TOO_SMALL (workspace), Q4NX_ERR_HIP.
 */
q4nx_status q4nx_flowkv_decode(const uint16_t* d_q, const uint16_t* d_k, const uint16_t* d_v, int64_t H, int64_t G,
                               int64_t d, int64_t L, int64_t t, int64_t window, float scale, void* d_o,
                               q4nx_dtype o_dtype, void* d_work, size_t work_bytes, hipStream_t stream);

/*
 * Device.  q4nx_flowkv_decode for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same computation and the same kernels -- so the same
 * bits -- with the chunk partials kept in the library's own static device
 * array of Q4NX_FLOWKV_STATIC_BYTES (16 MiB) per device instead of a caller
 * workspace.  Arguments as q4nx_flowkv_decode, without d_work/work_bytes.
 * The array is held by every device the library runs on until the process
 * ends; it is set up on the first call on each device (no allocation, no
 * synchronization).  Every call on one device shares that device's array:
 * calls that overlap on one device (concurrent streams, or host threads)
 * race and give wrong results; calls in one stream order are safe.  Nothing
 * in the array needs to start at zero (each call writes every partial it
 * reads).  Errors: as q4nx_flowkv_decode; Q4NX_ERR_BUFFER_TOO_SMALL when the
 * partials of the attended range, H * ceil(n / chunk) * (d + 4) * 4 bytes
 * (chunk = the launch's chunk length, 16-512), exceed the array -- e.g. the
 * Gemma3-27B geometry (H = 32, d = 128) up to about 64K attended positions
 * at any chunk length; Q4NX_ERR_HIP if the array cannot be located.
 */
#define Q4NX_FLOWKV_STATIC_BYTES ((size_t)16 << 20)
q4nx_status q4nx_flowkv_decode_static(const uint16_t* d_q, const uint16_t* d_k, const uint16_t* d_v, int64_t H,
                                      int64_t G, int64_t d, int64_t L, int64_t t, int64_t window, float scale,
                                      void* d_o, q4nx_dtype o_dtype, hipStream_t stream);

/*
 * The matrix product of q4nx_gemm, q4nx_mx_gemm and q4nx_gemm_bf16, with an
 * optional caller workspace (Sec. 3.1.2's tiled MM; the split along K is this
 * library's scheduling, not the paper's).
 *
 * w_format:  which of the three weight operands d_W is (a Q4NX blob, an
 *            MXFP4-variant blob, or bf16 [N][K]); other arguments as there.
 * d_work:    NULL, or device memory of at least
 *            q4nx_gemm_workspace_size(w_format, M, N, K) bytes (16-byte
 *            aligned), owned by the caller and used only while the call's
 *            launches run on `stream`; calls that overlap on one workspace
 *            race.
 * With a workspace the launch plan may split K for shapes with few output
 * tiles: each tile is then computed as up to 4 K segments whose float32
 * partial products are added in segment order by a second launch, so results
 * are deterministic but may differ in the last bits from the unsplit
 * product.  For Q4NX weights and a large M it may also dequantize W to bf16
 * in the workspace first (each weight once instead of once per row of output
 * tiles) and run the same plan on those weights, which gives the same bits as
 * the fused kernel.  With d_work == NULL nothing is split or staged and the
 * result equals the matching entry point's bit for bit.  Errors: as
 * q4nx_gemm; Q4NX_ERR_BUFFER_TOO_SMALL if work_bytes is below the need.
 */
typedef enum q4nx_weights {
  Q4NX_WEIGHTS_Q4NX = 0,
  Q4NX_WEIGHTS_MXFP4 = 1,
  Q4NX_WEIGHTS_BF16 = 2,
  Q4NX_WEIGHTS_RANGE_MIN_ = -2147483647 - 1, /* see q4nx_status */
  Q4NX_WEIGHTS_RANGE_MAX_ = 2147483647
} q4nx_weights;

/* Bytes of workspace q4nx_gemm_ex may use for (w_format, M, N, K) on the
 * current device (0 when it would use none, or if an argument is invalid). */
size_t q4nx_gemm_workspace_size(q4nx_weights w_format, int64_t M, int64_t N, int64_t K);

q4nx_status q4nx_gemm_ex(q4nx_weights w_format, int64_t M, int64_t N, int64_t K, const uint16_t* d_X,
                         const void* d_W, void* d_Y, q4nx_dtype y_dtype, void* d_work, size_t work_bytes,
                         hipStream_t stream);

/*
 * MXFP4 variant of the Q4NX block (the paper notes that Q4NX can be extended
 * to MXFP4, Sec. 3.1.1; element and scale encodings from the OCP Microscaling
 * (MX) specification v1.0): the same 32 x 256 blocks, strip-major order,
 * nibble layout and groups of 32 as Q4NX, with FP4 E2M1 codes (values 0, 0.5,
 * 1, 1.5, 2, 3, 4, 6, code bit 3 = sign) and one E8M0 scale byte per group,
 * X = 2^(e - 127), at index 8r + g after the codes -- 4352 bytes per block;
 * no offset.  w = X * fp4(q), exact in float32 and bf16.  Value domain of the
 * scales: e in [27, 227]; padding is code 0 with scale byte 127.
 */
size_t q4nx_mx_packed_size(int64_t N, int64_t K);  /* ceil(N/32)*ceil(K/256)*4352, 0 if invalid */

/* Host, synchronous: codes [N][K] (0..15) and E8M0 scales [N][K/32] -> blob.
 * Errors as q4nx_pack (a scale outside [27, 227] is Q4NX_ERR_INVALID_ARG). */
q4nx_status q4nx_mx_pack(const uint8_t* codes, const uint8_t* scales, int64_t N, int64_t K, void* blob,
                         size_t blob_bytes);

/* Host, synchronous: the inverse of q4nx_mx_pack. */
q4nx_status q4nx_mx_unpack(const void* blob, size_t blob_bytes, int64_t N, int64_t K, uint8_t* codes,
                           uint8_t* scales);

/* Device: float32 W [N][K] -> MXFP4-variant blob (the OCP MX v1.0 conversion):
 * per group the shared exponent e = floor(log2 max|w|) - 2, clamped to
 * [-100, 100] (0 for an all-zero group), and each element w / 2^e rounded to
 * the nearest FP4 value, ties to the even mantissa, saturating at 6.  Inputs
 * are first taken into the domain as by q4nx_quantize (NaN -> 0, clamp to
 * +-2^100), so every input gives a valid blob; padding is code 0 with scale
 * byte 127.  Arguments, alignment and errors as q4nx_quantize, with a blob of
 * q4nx_mx_packed_size(N, K) bytes. */
q4nx_status q4nx_mx_quantize(const float* d_W, int64_t N, int64_t K, void* d_blob, hipStream_t stream);

/* Device: q4nx_dequant for an MXFP4-variant blob (exact values; bf16 exact too). */
q4nx_status q4nx_mx_dequant(const void* d_blob, int64_t N, int64_t K, void* d_W, q4nx_dtype w_dtype,
                            hipStream_t stream);

/* Device: q4nx_gemv for an MXFP4-variant blob: y[n] = sum_k w[n][k] x[k] with the
 * same accumulation contract (float32, deterministic). */
q4nx_status q4nx_mx_gemv(const void* d_blob, const uint16_t* d_x, void* d_y, q4nx_dtype y_dtype, int64_t N,
                         int64_t K, hipStream_t stream);

/* Device: q4nx_gemv_batched for MXFP4-variant blobs (every descriptor's blob is one). */
q4nx_status q4nx_mx_gemv_batched(const q4nx_gemv_desc* descs, int32_t count, q4nx_dtype y_dtype,
                                 hipStream_t stream);

/* Device: q4nx_gemm for an MXFP4-variant blob (the bf16 weights are exact). */
q4nx_status q4nx_mx_gemm(int64_t M, int64_t N, int64_t K, const uint16_t* d_X, const void* d_blob, void* d_Y,
                         q4nx_dtype y_dtype, hipStream_t stream);

/* Measurement aid (not part of the projection path): reads `bytes` (a multiple
 * of 16, below 2^42) of device memory once with the GEMV's load pattern -- 2048
 * workgroups of 4 waves, workgroup b reading the b-th of 2048 equal contiguous
 * slices -- and writes 8192 floats to d_sink, which must hold them: float
 * 4b + w is the XOR of every 32-bit word wave w of workgroup b read (the
 * slice's 16-byte pieces p with p % 256 in [64w, 64w + 64)), masked to its low
 * 30 bits.  Timing it gives the read bandwidth, and the per-launch floor, of a
 * plain streaming kernel.  Device, asynchronous; errors as above (d_src
 * 16-byte aligned). */
q4nx_status q4nx_stream_read(const void* d_src, size_t bytes, float* d_sink, hipStream_t stream);

/* Static description of a status code. */
const char* q4nx_status_str(q4nx_status status);

/* Details of the last error reported on the calling thread ("" if none). */
const char* q4nx_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* Q4NX_H */
