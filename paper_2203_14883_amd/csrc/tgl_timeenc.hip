// tgl_timeenc.hip -- time encoding of sampled slots (Equation 3 of TGL: the
// time encoder of Section 2 maps a time difference dt to the vector
// cos(omega * dt + phi), omega and phi learnable vectors of the encoder's
// dimension).
//
// Each slot's row is dim independent elements, so the kernel is bound by the
// bytes it writes (dim * 4 or dim * 2 per slot against 4 read).  A wavefront
// encodes kRows slots at a time: one vector load brings their kRows time
// differences (lane u holds slot u's), each is broadcast from its lane, and
// lane l computes elements l, l + 64, ... of the row, so every store
// instruction writes 64 consecutive elements and no row waits on a load.
//
// Accuracy: the argument a = omega * dt + phi is formed in double precision
// (the product of two floats is exact there) and reduced in double to
// x = a - k pi/2 with |x| <= pi/4, before anything is rounded to float.  A
// plain float evaluation of the argument would be off by up to half an ulp of
// omega * dt -- 0.125 at dt = 2.7e6 s, Wikipedia's time span -- which the
// cosine passes on unchanged.  cos(a) is then +-cos(x) or +-sin(x) by the
// quadrant k mod 4, each from its Taylor series to the x^8 / x^9 term: on
// |x| <= pi/4 the first omitted terms are below 2.5e-8 and 2e-9, and the
// float Horner evaluation (fused multiply-adds) adds a few float ulps.  The
// result is within 1e-6 of cos(a).  Arguments of magnitude 2^31 or more,
// where the double reduction loses accuracy, use the double cosine instead.
//
// Padded slots (dt < 0) have no time difference: their rows are zeros, and a
// row's dt is the same for the whole wavefront, so those rows branch to plain
// stores.
#include "tgl_internal.hpp"

namespace tgl {
namespace {

constexpr int kRows = 16;                                          // slots per wavefront pass
constexpr double kTwoOverPi = 0.63661977236758134307553505349006;
constexpr double kPiOver2 = 1.5707963267948966192313216916398;

__device__ __forceinline__ float encode(float w, float dt, float ph) {
    const double a = fma(static_cast<double>(w), static_cast<double>(dt), static_cast<double>(ph));
    if (!(fabs(a) < 0x1p31)) return static_cast<float>(cos(a));  // huge, infinite or NaN arguments
    const double k = rint(a * kTwoOverPi);
    const float x = static_cast<float>(fma(-k, kPiOver2, a));      // |x| <= pi/4 up to rounding
    const float x2 = x * x;
    // Taylor series of cos and sin about 0, Horner form
    float c = __builtin_fmaf(x2, 1.0f / 40320.0f, -1.0f / 720.0f);
    c = __builtin_fmaf(x2, c, 1.0f / 24.0f);
    c = __builtin_fmaf(x2, c, -0.5f);
    c = __builtin_fmaf(x2, c, 1.0f);
    float sn = __builtin_fmaf(x2, 1.0f / 362880.0f, -1.0f / 5040.0f);
    sn = __builtin_fmaf(x2, sn, 1.0f / 120.0f);
    sn = __builtin_fmaf(x2, sn, -1.0f / 6.0f);
    sn = __builtin_fmaf(x2, sn, 1.0f);
    sn *= x;
    // cos(x + k pi/2) = cos x, -sin x, -cos x, sin x for k = 0, 1, 2, 3 mod 4
    const int q = static_cast<int>(static_cast<int64_t>(k) & 3);
    const float v = (q & 1) ? sn : c;
    return (q == 1 || q == 2) ? -v : v;
}

// float -> bfloat16, round to nearest even (NaN stays a quiet NaN)
__device__ __forceinline__ uint16_t to_bf16(float v) {
    const uint32_t b = __float_as_uint(v);
    if ((b & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((b >> 16) | 0x40u);
    return static_cast<uint16_t>((b + 0x7fffu + ((b >> 16) & 1u)) >> 16);
}

template <int OUT>
__global__ __launch_bounds__(kBlock) void timeenc_kernel(const float *__restrict__ dt, int64_t n,
                                                         const int64_t *__restrict__ count, int64_t per,
                                                         const float *__restrict__ omega,
                                                         const float *__restrict__ phi, int dim,
                                                         void *__restrict__ out) {
    const int lane = lane_id();
    constexpr int kWaves = kBlock / kWave;
    const int64_t waves = static_cast<int64_t>(gridDim.x) * kWaves;
    const int64_t wave = __builtin_amdgcn_readfirstlane(static_cast<int>(blockIdx.x * kWaves + threadIdx.x / kWave));
    if (count) {
        // valid prefix: min(n, count * per), without overflowing the product
        const int64_t c = *count;
        const int64_t lim = c <= 0 ? 0 : (c > n / per ? n : c * per);
        n = lim < n ? lim : n;
    }
    for (int64_t r0 = wave * kRows; r0 < n; r0 += waves * kRows) {
        const float dl = lane < kRows && r0 + lane < n ? dt[r0 + lane] : -1.0f;
#pragma unroll 1
        for (int u = 0; u < kRows; u++) {
            const int64_t row = r0 + u;
            if (row >= n) break;                                   // wavefront-uniform
            const float d = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, dl), u));
            const int64_t base = row * dim;
            if (d >= 0.0f) {                                       // wavefront-uniform
                for (int j = lane; j < dim; j += kWave) {
                    const float v = encode(omega[j], d, phi[j]);
                    if constexpr (OUT == TGL_OUT_F32)
                        __builtin_nontemporal_store(v, static_cast<float *>(out) + base + j);
                    else
                        __builtin_nontemporal_store(to_bf16(v), static_cast<uint16_t *>(out) + base + j);
                }
            } else {
                for (int j = lane; j < dim; j += kWave) {
                    if constexpr (OUT == TGL_OUT_F32)
                        __builtin_nontemporal_store(0.0f, static_cast<float *>(out) + base + j);
                    else
                        __builtin_nontemporal_store(static_cast<uint16_t>(0), static_cast<uint16_t *>(out) + base + j);
                }
            }
        }
    }
}

// Rows whose byte size is a multiple of 16: lane l of a wavefront owns the
// 16-byte word w0 + l of the flattened output (EPW elements: 4 float32 or 8
// bfloat16), so one store instruction writes 1 KB of contiguous output.  The
// word's row and column come from one 32-bit division by the uniform number
// of words per row.
template <int OUT>
__global__ __launch_bounds__(kBlock) void timeenc_vec_kernel(const float *__restrict__ dt, int64_t n,
                                                             const int64_t *__restrict__ count, int64_t per,
                                                             const float *__restrict__ omega,
                                                             const float *__restrict__ phi, int dim,
                                                             void *__restrict__ out) {
    constexpr int EPW = OUT == TGL_OUT_F32 ? 4 : 8;                 // elements per 16-byte word
    const int lane = lane_id();
    constexpr int kWaves = kBlock / kWave;
    const int64_t waves = static_cast<int64_t>(gridDim.x) * kWaves;
    const int64_t wave = __builtin_amdgcn_readfirstlane(static_cast<int>(blockIdx.x * kWaves + threadIdx.x / kWave));
    if (count) {
        const int64_t c = *count;
        const int64_t lim = c <= 0 ? 0 : (c > n / per ? n : c * per);
        n = lim < n ? lim : n;
    }
    const uint32_t wpr = static_cast<uint32_t>(dim / EPW);           // words per row
    const int64_t total = n * wpr;
    int4 *const o = static_cast<int4 *>(out);
    for (int64_t w0 = wave * kWave; w0 < total; w0 += waves * kWave) {
        const int64_t row0 = w0 / wpr;                                // wavefront-uniform
        const uint32_t r = static_cast<uint32_t>(w0 - row0 * wpr) + static_cast<uint32_t>(lane);
        const uint32_t dr = r / wpr;
        const int64_t row = row0 + dr;
        const int col = static_cast<int>(r - dr * wpr) * EPW;
        if (w0 + lane >= total) continue;
        const float d = dt[row];
        float v[EPW];
        if (d >= 0.0f) {
#pragma unroll
            for (int e = 0; e < EPW; e++) v[e] = encode(omega[col + e], d, phi[col + e]);
        } else {
#pragma unroll
            for (int e = 0; e < EPW; e++) v[e] = 0.0f;
        }
        int4 word;
        if constexpr (OUT == TGL_OUT_F32) {
            word = make_int4(__float_as_int(v[0]), __float_as_int(v[1]), __float_as_int(v[2]), __float_as_int(v[3]));
        } else {
            uint32_t pk[4];
#pragma unroll
            for (int e = 0; e < 4; e++)
                pk[e] = static_cast<uint32_t>(to_bf16(v[2 * e])) | (static_cast<uint32_t>(to_bf16(v[2 * e + 1])) << 16);
            word = make_int4(static_cast<int>(pk[0]), static_cast<int>(pk[1]), static_cast<int>(pk[2]),
                             static_cast<int>(pk[3]));
        }
        o[w0 + lane] = word;
    }
}

}  // namespace
}  // namespace tgl

using namespace tgl;

extern "C" {

tgl_status tgl_time_encode(const float *dt, int64_t n, const int64_t *count, int64_t per_count,
                           const float *omega, const float *phi, int32_t dim, int32_t out_type,
                           void *out, void *stream) {
    if (n < 0 || per_count < 1 || dim < 1 || dim > TGL_MAX_TIME_DIM) return TGL_EINVAL;
    if (out_type != TGL_OUT_F32 && out_type != TGL_OUT_BF16) return TGL_EINVAL;
    if (!omega || !phi) return TGL_EINVAL;
    if (n > 0 && (!dt || !out)) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(out) & 3u) != 0) return TGL_EINVAL;
    if (n > INT64_MAX / dim) return TGL_EINVAL;
    if (n == 0) return TGL_OK;
    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    const int esize = out_type == TGL_OUT_F32 ? 4 : 2;
    const bool vec = (static_cast<int64_t>(dim) * esize) % 16 == 0 && (reinterpret_cast<uintptr_t>(out) & 15u) == 0;
    if (vec) {
        const int64_t words = n * (static_cast<int64_t>(dim) * esize / 16);
        int64_t blocks = (words + kBlock - 1) / kBlock;
        if (blocks > (1 << 16)) blocks = 1 << 16;
        ScopedTimer tm(TGL_TIMER_TIMEENC, st);
        if (out_type == TGL_OUT_F32)
            timeenc_vec_kernel<TGL_OUT_F32><<<static_cast<unsigned>(blocks), kBlock, 0, st>>>(
                dt, n, count, per_count, omega, phi, dim, out);
        else
            timeenc_vec_kernel<TGL_OUT_BF16><<<static_cast<unsigned>(blocks), kBlock, 0, st>>>(
                dt, n, count, per_count, omega, phi, dim, out);
        return launch_status();
    }
    constexpr int64_t rows_per_block = static_cast<int64_t>(kBlock / kWave) * kRows;
    int64_t blocks = (n + rows_per_block - 1) / rows_per_block;
    if (blocks > (1 << 16)) blocks = 1 << 16;
    {
        ScopedTimer tm(TGL_TIMER_TIMEENC, st);
        if (out_type == TGL_OUT_F32)
            timeenc_kernel<TGL_OUT_F32><<<static_cast<unsigned>(blocks), kBlock, 0, st>>>(dt, n, count, per_count,
                                                                                         omega, phi, dim, out);
        else
            timeenc_kernel<TGL_OUT_BF16><<<static_cast<unsigned>(blocks), kBlock, 0, st>>>(dt, n, count, per_count,
                                                                                          omega, phi, dim, out);
    }
    return launch_status();
}

}  // extern "C"
