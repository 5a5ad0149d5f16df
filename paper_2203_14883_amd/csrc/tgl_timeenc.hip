// tgl_timeenc.hip -- time encoding of sampled slots (Equation 3 of TGL: the
// time encoder of Section 2 maps a time difference dt to the vector
// cos(omega * dt + phi), omega and phi learnable vectors of the encoder's
// dimension).
//
// Each slot's row is dim independent elements, so the kernel is bound by the
// bytes it writes (dim * 4 or dim * 2 per slot against 4 read).  A wavefront
// encodes kRows slots at a time, lane l computing elements l, l + 64, ... of
// each row, so every store instruction writes 64 consecutive elements.
//
// Accuracy: the argument omega * dt + phi is formed in double precision (the
// product of two floats is exact there), reduced modulo 2 pi in double, and
// only then rounded to float for the float cosine.  The float argument a
// straightforward float evaluation would use is off by up to half an ulp of
// omega * dt -- 0.125 at dt = 2.7e6 s, Wikipedia's time span -- which the
// cosine passes on unchanged.
#include "tgl_internal.hpp"

namespace tgl {
namespace {

constexpr int kRows = 4;                                           // slots per wavefront pass
constexpr double kTwoPi = 6.283185307179586476925286766559;
constexpr double kInvTwoPi = 0.15915494309189533576888376337251;

__device__ __forceinline__ float encode(float w, float dt, float ph) {
    const double a = fma(static_cast<double>(w), static_cast<double>(dt), static_cast<double>(ph));
    const double k = rint(a * kInvTwoPi);
    const double r = fma(-k, kTwoPi, a);                           // in [-pi, pi] up to rounding
    return cosf(static_cast<float>(r));
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
        float d[kRows];
#pragma unroll
        for (int u = 0; u < kRows; u++) d[u] = r0 + u < n ? dt[r0 + u] : -1.0f;
        for (int j = lane; j < dim; j += kWave) {
            const float w = omega[j];
            const float ph = phi[j];
#pragma unroll
            for (int u = 0; u < kRows; u++) {
                const int64_t row = r0 + u;
                if (row >= n) continue;
                const float v = d[u] >= 0.0f ? encode(w, d[u], ph) : 0.0f;
                const int64_t o = row * dim + j;
                if constexpr (OUT == TGL_OUT_F32)
                    __builtin_nontemporal_store(v, static_cast<float *>(out) + o);
                else
                    __builtin_nontemporal_store(to_bf16(v), static_cast<uint16_t *>(out) + o);
            }
        }
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
