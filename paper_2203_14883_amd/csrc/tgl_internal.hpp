// tgl_internal.hpp -- helpers shared by the libtgl translation units:
// launch checking, kernel timers, wave-level primitives and the device-wide
// exclusive scan used by both the T-CSR build and the sampler.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tgl.h"

namespace tgl {

constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kBlock = 256;        // threads per block for every kernel here
constexpr int kScanItems = 8;      // items per thread in the scan kernels
constexpr int kScanTile = kBlock * kScanItems;

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Bump allocator over a caller-provided workspace (or a dry run when base is
// null, to compute the size).
struct Carver {
    char *base;
    size_t off = 0;
    explicit Carver(void *b) : base(static_cast<char *>(b)) {}
    template <class T>
    T *take(size_t count) {
        off = align_up(off, 256);
        T *p = base ? reinterpret_cast<T *>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
    size_t size() const { return align_up(off, 256); }
};

// ---- kernel timers (implemented in tgl_runtime.hip) ----
int timer_begin(int kind, hipStream_t s);    // returns a slot or -1
void timer_end(int slot, hipStream_t s);

struct ScopedTimer {
    int slot;
    hipStream_t s;
    ScopedTimer(int kind, hipStream_t st) : slot(timer_begin(kind, st)), s(st) {}
    ~ScopedTimer() { timer_end(slot, s); }
};

inline tgl_status launch_status() {
    return hipGetLastError() == hipSuccess ? TGL_OK : TGL_EDEVICE;
}

// ---- wave-level primitives ----

__device__ __forceinline__ int lane_id() { return static_cast<int>(threadIdx.x & (kWave - 1)); }

// Number of set bits of a wave-wide mask below the calling lane.
__device__ __forceinline__ int rank_below(uint64_t mask) {
    return static_cast<int>(__builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                                      __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u)));
}

// Ballot restricted to the G-lane group of the calling lane (bit i = lane i
// of the group).  Lanes of one group must be active together.
template <int G>
__device__ __forceinline__ uint64_t group_ballot(bool pred) {
    const uint64_t m = __ballot(pred);
    if constexpr (G == kWave) {
        return m;
    } else {
        const int shift = lane_id() & ~(G - 1);
        return (m >> shift) & ((1ull << G) - 1ull);
    }
}

// Inclusive prefix sum over the 64 lanes of a wave.
template <class T>
__device__ __forceinline__ T wave_inclusive_sum(T v) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
        const T o = __shfl_up(v, d, kWave);
        if (lane_id() >= d) v += o;
    }
    return v;
}

// Exclusive prefix sum over a 256-thread block; returns the block total in
// *total.  `lds` must hold kBlock / kWave elements.
template <class T>
__device__ __forceinline__ T block_exclusive_sum(T v, T *lds, T *total) {
    const T inc = wave_inclusive_sum(v);
    const int w = threadIdx.x / kWave;
    if (lane_id() == kWave - 1) lds[w] = inc;
    __syncthreads();
    T before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < kBlock / kWave; i++) {
        const T x = lds[i];
        if (i < w) before += x;
        all += x;
    }
    __syncthreads();
    *total = all;
    return before + inc - v;
}

// ---- device-wide exclusive scan (reduce, scan partials, apply) ----
//
// in[0..n) -> out[0..n), n = *n_dyn when n_dyn is not null (read on the
// device, so the length can come from an earlier kernel), else n_static.
// Tiles of kScanTile items; `partials` holds one int64 per tile.

template <class TIn>
__global__ __launch_bounds__(kBlock) void scan_reduce_kernel(const TIn *__restrict__ in,
                                                              int64_t n_static,
                                                              const int64_t *__restrict__ n_dyn,
                                                              int64_t *__restrict__ partials) {
    __shared__ int64_t lds[kBlock / kWave];
    const int64_t n = n_dyn ? *n_dyn : n_static;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile;
    int64_t sum = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; i++) {
        const int64_t idx = base + static_cast<int64_t>(i) * kBlock + threadIdx.x;
        if (idx < n) sum += static_cast<int64_t>(in[idx]);
    }
    int64_t total;
    block_exclusive_sum<int64_t>(sum, lds, &total);
    if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

// Launches one block of 1024 threads that turns partials[0..nb) into
// exclusive offsets and stores the grand total in *total_out (if not null).
// Defined in tgl_runtime.hip.
void launch_scan_partials(int64_t *partials, int64_t nb, int64_t *total_out, hipStream_t s);

template <class TIn, class TOut>
__global__ __launch_bounds__(kBlock) void scan_apply_kernel(const TIn *__restrict__ in,
                                                             TOut *__restrict__ out,
                                                             int64_t n_static,
                                                             const int64_t *__restrict__ n_dyn,
                                                             const int64_t *__restrict__ partials) {
    __shared__ int64_t lds[kBlock / kWave];
    const int64_t n = n_dyn ? *n_dyn : n_static;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile +
                         static_cast<int64_t>(threadIdx.x) * kScanItems;
    int64_t v[kScanItems];
    int64_t sum = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; i++) {
        const int64_t idx = base + i;
        v[i] = idx < n ? static_cast<int64_t>(in[idx]) : 0;
        sum += v[i];
    }
    int64_t total;
    int64_t run = block_exclusive_sum<int64_t>(sum, lds, &total) + partials[blockIdx.x];
#pragma unroll
    for (int i = 0; i < kScanItems; i++) {
        const int64_t idx = base + i;
        if (idx < n) out[idx] = static_cast<TOut>(run);
        run += v[i];
    }
}

inline int64_t scan_tiles(int64_t n) { return (n + kScanTile - 1) / kScanTile; }

}  // namespace tgl
