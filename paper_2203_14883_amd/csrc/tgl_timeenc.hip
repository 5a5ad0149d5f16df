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
// Accuracy: the argument is formed in turns, t = (omega / 2 pi) dt + phi / 2 pi,
// in double precision, from per-column factors omega / 2 pi and phi / 2 pi
// (each within 2^-52 relative of exact); below 2^24 turns t is within 5e-8
// rad of the exact argument.  Its fraction f = t - rint(t) is exact, and
// cos(2 pi f) = cos(2 pi g) for g = |f| in [0, 1/2]; above 1/4 it is
// -cos(2 pi (1/2 - g)), also exact, so only [0, 1/4] is left: x = 2 pi g
// in [0, pi/2], where the cosine's Taylor series to x^12, in powers of g^2,
// leaves out less than 6.4e-9.  g is rounded to float (2.4e-8 rad) and the
// series evaluated by fused multiply-adds in float (a few float ulps).  The
// result is within 3e-7 of cos(omega dt + phi).  A plain float evaluation of
// the argument would be off by up to half an ulp of omega * dt -- 0.125 at
// dt = 2.7e6 s, Wikipedia's time span -- which the cosine passes on
// unchanged.  Arguments of 2^24 turns or more, infinite or NaN use the double
// cosine of the double argument instead.
//
// Padded slots (dt < 0) have no time difference: their rows are zeros, and a
// row's dt is the same for the whole wavefront, so those rows branch to plain
// stores.
#include <atomic>

#include "tgl_internal.hpp"

namespace tgl {
namespace {

constexpr int kRows = 16;                                          // slots per wavefront pass
constexpr double kInvTwoPi = 0.15915494309189535;                  // 1 / (2 pi), nearest double
constexpr double kTurnLimit = 0x1p24;                              // turns reduced in double below this
constexpr int kMaxPre = 1024;                                      // columns whose factors fit in LDS

// cos(2 pi g) = sum_n c_n g^(2n), c_n = (-1)^n (2 pi)^(2n) / (2n)!  (n <= 6)
constexpr float kC1 = -19.739208802178717f;
constexpr float kC2 = 64.93939402266829f;
constexpr float kC3 = -85.45681720669373f;
constexpr float kC4 = 60.24464137187666f;
constexpr float kC5 = -26.426256783374397f;
constexpr float kC6 = 7.903536371318469f;

// cos(2 pi t) for an argument t in turns with |t| < kTurnLimit
__device__ __forceinline__ float cos_turns(double t) {
    const double f = t - rint(t);                                  // exact, in [-1/2, 1/2]
    const double a = fabs(f);
    const bool flip = a > 0.25;                                    // cos(2 pi a) = -cos(2 pi (1/2 - a))
    const float g = static_cast<float>(fmin(a, 0.5 - a));         // 0.5 - a is exact; flip picks it
    const float y = g * g;
    float c = __builtin_fmaf(y, kC6, kC5);
    c = __builtin_fmaf(y, c, kC4);
    c = __builtin_fmaf(y, c, kC3);
    c = __builtin_fmaf(y, c, kC2);
    c = __builtin_fmaf(y, c, kC1);
    c = __builtin_fmaf(y, c, 1.0f);
    return flip ? -c : c;
}

// cos(omega dt + phi) from wp = omega / 2 pi and pp = phi / 2 pi; omega[j] and
// phi[j] are read only for the double-precision fallback.
__device__ __forceinline__ float encode(double wp, double pp, float dt, const float *__restrict__ omega,
                                        const float *__restrict__ phi, int j) {
    const double t = fma(wp, static_cast<double>(dt), pp);        // the argument in turns
    if (!(fabs(t) < kTurnLimit))                                   // huge, infinite or NaN
        return static_cast<float>(cos(fma(static_cast<double>(omega[j]), static_cast<double>(dt),
                                          static_cast<double>(phi[j]))));
    return cos_turns(t);
}

// the per-column factors (omega / 2 pi, phi / 2 pi) of columns [0, dim), into
// LDS by the whole block (dim <= kMaxPre)
__device__ __forceinline__ void load_factors(double2 *__restrict__ f, const float *__restrict__ omega,
                                             const float *__restrict__ phi, int dim) {
    for (int j = threadIdx.x; j < dim; j += kBlock)
        f[j] = make_double2(static_cast<double>(omega[j]) * kInvTwoPi, static_cast<double>(phi[j]) * kInvTwoPi);
    __syncthreads();
}

// float -> bfloat16, round to nearest even (NaN stays a quiet NaN)
__device__ __forceinline__ uint16_t to_bf16(float v) {
    const uint32_t b = __float_as_uint(v);
    if ((b & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((b >> 16) | 0x40u);
    return static_cast<uint16_t>((b + 0x7fffu + ((b >> 16) & 1u)) >> 16);
}

template <int OUT, bool PRE>
__global__ __launch_bounds__(kBlock) void timeenc_kernel(const float *__restrict__ dt, int64_t n,
                                                         const int64_t *__restrict__ count, int64_t per,
                                                         const float *__restrict__ omega,
                                                         const float *__restrict__ phi, int dim,
                                                         void *__restrict__ out) {
    __shared__ double2 fac[PRE ? kMaxPre : 1];
    if constexpr (PRE) load_factors(fac, omega, phi, dim);
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
                    const double2 fj = PRE ? fac[j]
                                           : make_double2(static_cast<double>(omega[j]) * kInvTwoPi,
                                                          static_cast<double>(phi[j]) * kInvTwoPi);
                    const float v = encode(fj.x, fj.y, d, omega, phi, j);
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
// bfloat16), so one store instruction writes 1 KB of contiguous output.
// With float32 output and the factors in LDS, a lane reads its word's four
// factor pairs together and checks the four arguments once, so the elements
// are evaluated side by side rather than each behind its own LDS wait and
// branch; that kernel is held to 64 VGPRs, i.e. 8 wavefronts per SIMD (at 7
// it is slower than the element-by-element form).  The other forms keep the
// element-by-element evaluation, which needs fewer registers.
template <int OUT, bool PRE>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(OUT == TGL_OUT_F32 && PRE ? 8 : 1)))
void timeenc_vec_kernel(const float *__restrict__ dt, int64_t n, const int64_t *__restrict__ count, int64_t per,
                        const float *__restrict__ omega, const float *__restrict__ phi, int dim,
                        void *__restrict__ out) {
    constexpr int EPW = OUT == TGL_OUT_F32 ? 4 : 8;                 // elements per 16-byte word
    __shared__ double2 fac[PRE ? kMaxPre : 1];
    if constexpr (PRE) load_factors(fac, omega, phi, dim);
    const int lane = lane_id();
    constexpr int kWaves = kBlock / kWave;
    const int64_t waves = static_cast<int64_t>(gridDim.x) * kWaves;
    const int64_t wave = __builtin_amdgcn_readfirstlane(static_cast<int>(blockIdx.x * kWaves + threadIdx.x / kWave));
    if (count) {
        const int64_t c = *count;
        const int64_t lim = c <= 0 ? 0 : (c > n / per ? n : c * per);
        n = lim < n ? lim : n;
    }
    const uint32_t wpr = static_cast<uint32_t>(dim / EPW);           // words per row, at most 1024
    const int64_t total = n * wpr;
    int4 *const o = static_cast<int4 *>(out);
    // The wavefront's first word w0 as (row0, off0), advanced by the grid
    // stride without dividing; a lane's word w0 + lane is off0 + lane < wpr + 64
    // words past row0's start, split by a float reciprocal (exact after one
    // correction: the quotient is at most 64 and the product is within 2^-22
    // of it).
    const float inv_wpr = 1.0f / static_cast<float>(wpr);
    const int64_t step = waves * kWave;
    const int64_t step_q = step / wpr;
    const uint32_t step_r = static_cast<uint32_t>(step - step_q * wpr);
    int64_t w0 = wave * kWave;
    int64_t row0 = w0 / wpr;
    uint32_t off0 = static_cast<uint32_t>(w0 - row0 * wpr);
    for (; w0 < total; w0 += step) {
        if (w0 + lane < total) {
            const uint32_t r = off0 + static_cast<uint32_t>(lane);
            uint32_t dr = static_cast<uint32_t>(static_cast<float>(r) * inv_wpr);
            if ((dr + 1) * wpr <= r) dr++;
            const int64_t row = row0 + dr;
            const int col = static_cast<int>(r - dr * wpr) * EPW;
            const float d = dt[row];
            float v[EPW];
            if (d < 0.0f) {
#pragma unroll
                for (int e = 0; e < EPW; e++) v[e] = 0.0f;
            } else if constexpr (OUT == TGL_OUT_F32 && PRE) {
                // the factors as the general form reads them: with a plain
                // fac[col + e] hipcc combines the four range checks through
                // 16-bit vector ops instead of lane masks, and runs slower
                double2 fj[EPW];
#pragma unroll
                for (int e = 0; e < EPW; e++)
                    fj[e] = PRE ? fac[col + e]
                                : make_double2(static_cast<double>(omega[col + e]) * kInvTwoPi,
                                               static_cast<double>(phi[col + e]) * kInvTwoPi);
                const double dd = static_cast<double>(d);
                double t[EPW];
                bool ok = true;
#pragma unroll
                for (int e = 0; e < EPW; e++) {
                    t[e] = fma(fj[e].x, dd, fj[e].y);
                    ok = ok && fabs(t[e]) < kTurnLimit;
                }
                if (ok) {                           // the arguments encode() reduces itself
#pragma unroll
                    for (int e = 0; e < EPW; e++) v[e] = cos_turns(t[e]);
                } else {
#pragma unroll
                    for (int e = 0; e < EPW; e++) v[e] = encode(fj[e].x, fj[e].y, d, omega, phi, col + e);
                }
            } else {
#pragma unroll
                for (int e = 0; e < EPW; e++) {
                    const double2 fj = PRE ? fac[col + e]
                                           : make_double2(static_cast<double>(omega[col + e]) * kInvTwoPi,
                                                          static_cast<double>(phi[col + e]) * kInvTwoPi);
                    v[e] = encode(fj.x, fj.y, d, omega, phi, col + e);
                }
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
        row0 += step_q;
        off0 += step_r;
        if (off0 >= wpr) {
            off0 -= wpr;
            row0++;
        }
    }
}

// Both kernels stride over their rows, so a grid of the blocks the device
// holds at once does all the work and loads each block's factor table once:
// with one block per 256 words (capped at 64 Ki blocks) a block lived for
// about a dozen words and its factor load and barrier were a tenth of its
// time.  Found once per device and kernel (CUs x resident blocks per CU).
constexpr int kMaxDevices = 64;
constexpr int kVariants = 8;                                       // row/word kernel x output x factor table
std::atomic<int> g_resident[kMaxDevices][kVariants];

template <typename K>
unsigned resident_grid(K kernel, int variant, int64_t want) {
    int dev = 0;
    int r = 0;
    if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < kMaxDevices) {
        r = g_resident[dev][variant].load(std::memory_order_relaxed);
        if (r == 0) {
            int cus = 0, per_cu = 0;
            if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
                hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kBlock, 0) == hipSuccess && cus > 0 &&
                per_cu > 0) {
                r = cus * per_cu;
                g_resident[dev][variant].store(r, std::memory_order_relaxed);
            }
        }
    }
    (void)hipGetLastError();
    if (r <= 0) r = 1 << 16;
    return static_cast<unsigned>(want < r ? want : r);
}

template <typename K>
void launch_resident(K kernel, int variant, int64_t want, hipStream_t st, const float *dt, int64_t n,
                     const int64_t *count, int64_t per, const float *omega, const float *phi, int dim, void *out) {
    const unsigned nb = resident_grid(kernel, variant, want);
    ScopedTimer tm(TGL_TIMER_TIMEENC, st);
    kernel<<<nb, kBlock, 0, st>>>(dt, n, count, per, omega, phi, dim, out);
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
    const bool pre = dim <= kMaxPre;                      // per-column factors staged in LDS
    const bool vec = (static_cast<int64_t>(dim) * esize) % 16 == 0 && (reinterpret_cast<uintptr_t>(out) & 15u) == 0;
    if (vec) {
        const int64_t words = n * (static_cast<int64_t>(dim) * esize / 16);
        const int64_t want = (words + kBlock - 1) / kBlock;
        if (out_type == TGL_OUT_F32) {
            if (pre) launch_resident(timeenc_vec_kernel<TGL_OUT_F32, true>, 4, want, st, dt, n, count, per_count, omega, phi, dim, out);
            else launch_resident(timeenc_vec_kernel<TGL_OUT_F32, false>, 5, want, st, dt, n, count, per_count, omega, phi, dim, out);
        } else {
            if (pre) launch_resident(timeenc_vec_kernel<TGL_OUT_BF16, true>, 6, want, st, dt, n, count, per_count, omega, phi, dim, out);
            else launch_resident(timeenc_vec_kernel<TGL_OUT_BF16, false>, 7, want, st, dt, n, count, per_count, omega, phi, dim, out);
        }
        return launch_status();
    }
    constexpr int64_t rows_per_block = static_cast<int64_t>(kBlock / kWave) * kRows;
    const int64_t want = (n + rows_per_block - 1) / rows_per_block;
    if (out_type == TGL_OUT_F32) {
        if (pre) launch_resident(timeenc_kernel<TGL_OUT_F32, true>, 0, want, st, dt, n, count, per_count, omega, phi, dim, out);
        else launch_resident(timeenc_kernel<TGL_OUT_F32, false>, 1, want, st, dt, n, count, per_count, omega, phi, dim, out);
    } else {
        if (pre) launch_resident(timeenc_kernel<TGL_OUT_BF16, true>, 2, want, st, dt, n, count, per_count, omega, phi, dim, out);
        else launch_resident(timeenc_kernel<TGL_OUT_BF16, false>, 3, want, st, dt, n, count, per_count, omega, phi, dim, out);
    }
    return launch_status();
}

}  // extern "C"
