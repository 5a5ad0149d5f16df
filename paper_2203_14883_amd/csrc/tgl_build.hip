// tgl_build.hip -- T-CSR build (Section 3.1, "The T-CSR Data Structure").
//
// Every directed entry i gets a 64-bit sort key holding its owner node and
// its timestamp (as tskey, an unsigned integer with the float order); a
// stable least-significant-digit radix sort of (key, i) then leaves each
// node's entries contiguous and sorted by (ts, i), which is the T-CSR order.
// A first pass validates the edges and OR- and AND-reduces node ids and
// tskeys, so bits on which every entry agrees are known before any key is
// written.  When the varying node bits, the varying tskey bits and the
// neighbour id fit in 64 bits together (c4: 27 + 8 + 27), a key packs them in
// that order: the sort runs over the node and tskey fields only (five 8-bit
// passes for c4 instead of six), and the neighbour id rides in the low bits,
// so writing the entries reads the sorted keys and indices in order instead
// of gathering each neighbour by original edge index.  Otherwise the key is
// (node << 32 | tskey) and the digits every key shares are skipped.  Each
// radix pass is reduce-then-scan: per-tile digit counts, a device-wide scan in
// digit-major order, and a scatter in which every wavefront ranks its keys
// with ballots (stable within the tile), the tile is reordered in LDS and
// written out bucket by bucket.
//
// The paper builds the T-CSR once on the host; here the same structure is
// produced on the device from a COO that may be in any order.
#include "tgl_cells.hpp"
#include "tgl_internal.hpp"

namespace tgl {
namespace {

constexpr int kMaxRadixBits = 8;                  // digits of 7 or 8 bits
constexpr int kBins = 1 << kMaxRadixBits;         // histogram rows per tile (the most digits can need)
constexpr int kTileItems = 16;                    // keys per thread per radix tile
constexpr int kTile = kBlock * kTileItems;        // 4096 keys
constexpr int kWaves = kBlock / kWave;
constexpr int kWaveTile = kTile / kWaves;         // 1024 keys per wavefront
constexpr int64_t kMaxEntries = (int64_t(1) << 32) - 1;
constexpr int kXcds = 8;                          // accelerator dies, each with its own L2

// Tile of block b in the radix kernels.  Workgroups are dealt to the dies
// round-robin, so block b runs on die b % 8; each die takes a contiguous
// range of tiles instead, so that neighbouring tiles -- which write adjacent
// counts of each histogram row and adjacent pieces of each digit's output
// run -- share one L2, where their partial lines merge.  Returns -1 for the
// blocks past the last tile (the grid is a multiple of 8).
__device__ __forceinline__ int64_t radix_tile(int64_t ntiles) {
    const int64_t per = (ntiles + kXcds - 1) / kXcds;
    const int64_t b = blockIdx.x;
    const int64_t t = (b % kXcds) * per + b / kXcds;
    return t < ntiles ? t : -1;
}

unsigned radix_grid(int64_t ntiles) {
    return static_cast<unsigned>((ntiles + kXcds - 1) / kXcds * kXcds);
}

struct BuildFlags {
    uint32_t err;
    uint32_t pad;
    uint64_t or_bits;
    uint64_t and_bits;
};

__device__ __forceinline__ uint32_t ts_key(float t) {
    const uint32_t b = __float_as_uint(t == 0.0f ? 0.0f : t);   // -0 -> +0
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float key_ts(uint32_t k) {
    const uint32_t b = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
    return __uint_as_float(b);
}

template <class T>
__device__ __forceinline__ T wave_or(T v) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) v |= __shfl_xor(v, d, kWave);
    return v;
}

template <class T>
__device__ __forceinline__ T wave_and(T v) {
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) v &= __shfl_xor(v, d, kWave);
    return v;
}

__global__ void init_flags_kernel(BuildFlags *f) {
    f->err = 0;
    f->pad = 0;
    f->or_bits = 0;
    f->and_bits = ~0ull;
}

// How a sort key holds (owner node, tskey, neighbour).  Packed: node field,
// tskey field, neighbour id, from the most significant bits down; a field
// keeps bits [lo, lo + bits) of its value, the bits outside being the same in
// every entry (konst).  Unpacked: node << 32 | tskey.
struct KeyLayout {
    int packed;
    int nbr_bits;
    int ts_lo, ts_bits;
    int node_lo, node_bits;
    uint32_t ts_konst, node_konst;
};

__host__ __device__ __forceinline__ uint64_t low_mask(int bits) {
    return bits >= 64 ? ~0ull : (1ull << bits) - 1ull;
}

__device__ __forceinline__ uint64_t make_key(const KeyLayout &L, uint32_t u, uint32_t tk, uint32_t v) {
    if (!L.packed) return (static_cast<uint64_t>(u) << 32) | tk;
    const uint64_t nf = (static_cast<uint64_t>(u) >> L.node_lo) & low_mask(L.node_bits);
    const uint64_t tf = (static_cast<uint64_t>(tk) >> L.ts_lo) & low_mask(L.ts_bits);
    return (nf << (L.nbr_bits + L.ts_bits)) | (tf << L.nbr_bits) | static_cast<uint64_t>(v);
}

__device__ __forceinline__ uint32_t key_node(const KeyLayout &L, uint64_t k) {
    if (!L.packed) return static_cast<uint32_t>(k >> 32);
    const uint64_t nf = (k >> (L.nbr_bits + L.ts_bits)) & low_mask(L.node_bits);
    return L.node_konst | static_cast<uint32_t>(nf << L.node_lo);
}

__device__ __forceinline__ uint32_t key_tskey(const KeyLayout &L, uint64_t k) {
    if (!L.packed) return static_cast<uint32_t>(k);
    const uint64_t tf = (k >> L.nbr_bits) & low_mask(L.ts_bits);
    return L.ts_konst | static_cast<uint32_t>(tf << L.ts_lo);
}

// Edges per thread and grid-stride round of the kernels that read the edge
// list: their loads are issued together, one coalesced stream per array.
constexpr int kEdgeUnroll = 4;

// Validation and the OR / AND of the node ids and tskeys of every entry (one
// read of each edge: both directions when undirected).  One set of atomics
// per block.
__global__ __launch_bounds__(kBlock) void reduce_kernel(const int32_t *__restrict__ src,
                                                        const int32_t *__restrict__ dst,
                                                        const float *__restrict__ ts, int64_t m0, bool both,
                                                        int64_t N, BuildFlags *__restrict__ flags) {
    __shared__ uint64_t s_or[kWaves], s_and[kWaves];
    __shared__ uint32_t s_bad[kWaves];
    uint64_t o = 0, a = ~0ull;
    bool bad = false;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock * kEdgeUnroll;
    for (int64_t k0 = static_cast<int64_t>(blockIdx.x) * kBlock * kEdgeUnroll + threadIdx.x; k0 < m0; k0 += stride) {
        int32_t u[kEdgeUnroll], v[kEdgeUnroll];
        float t[kEdgeUnroll];
#pragma unroll
        for (int j = 0; j < kEdgeUnroll; j++) {
            const int64_t k = k0 + static_cast<int64_t>(j) * kBlock;
            const bool in = k < m0;
            u[j] = in ? src[k] : 0;
            v[j] = in ? dst[k] : 0;
            t[j] = in ? ts[k] : 0.0f;
            if (!in) {   // neutral for the OR / AND: repeat a key that is present (edge k0)
                u[j] = u[0];
                v[j] = v[0];
                t[j] = t[0];
            }
        }
#pragma unroll
        for (int j = 0; j < kEdgeUnroll; j++) {
            bad |= u[j] < 0 || u[j] >= N || v[j] < 0 || v[j] >= N || t[j] != t[j];
            const uint64_t tk = ts_key(t[j]);
            const uint64_t ku = (static_cast<uint64_t>(static_cast<uint32_t>(u[j])) << 32) | tk;
            o |= ku;
            a &= ku;
            if (both) {
                const uint64_t kv = (static_cast<uint64_t>(static_cast<uint32_t>(v[j])) << 32) | tk;
                o |= kv;
                a &= kv;
            }
        }
    }
    o = wave_or(o);
    a = wave_and(a);
    const bool any_bad = __ballot(bad) != 0;
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0) {
        s_or[w] = o;
        s_and[w] = a;
        s_bad[w] = any_bad ? 1u : 0u;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t bb = 0;
#pragma unroll
        for (int i = 1; i < kWaves; i++) {
            o |= s_or[i];
            a &= s_and[i];
        }
#pragma unroll
        for (int i = 0; i < kWaves; i++) bb |= s_bad[i];
        atomicOr(reinterpret_cast<unsigned long long *>(&flags->or_bits), static_cast<unsigned long long>(o));
        atomicAnd(reinterpret_cast<unsigned long long *>(&flags->and_bits), static_cast<unsigned long long>(a));
        if (bb) atomicOr(&flags->err, 1u);
    }
}

// Entry k < m0: (src[k] -> dst[k]); entry m0 + k: (dst[k] -> src[k]) when
// undirected, written from the same read of edge k.  Keys in the layout L,
// values the entry indices.
__global__ __launch_bounds__(kBlock) void keys_kernel(const int32_t *__restrict__ src,
                                                      const int32_t *__restrict__ dst, const float *__restrict__ ts,
                                                      int64_t m0, bool both, const KeyLayout L,
                                                      uint64_t *__restrict__ keys, uint32_t *__restrict__ vals) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock * kEdgeUnroll;
    for (int64_t k0 = static_cast<int64_t>(blockIdx.x) * kBlock * kEdgeUnroll + threadIdx.x; k0 < m0; k0 += stride) {
        uint32_t u[kEdgeUnroll], v[kEdgeUnroll], tk[kEdgeUnroll];
#pragma unroll
        for (int j = 0; j < kEdgeUnroll; j++) {
            // clamped, not predicated, so that the loads issue back to back
            const int64_t k = k0 + static_cast<int64_t>(j) * kBlock;
            const int64_t kc = k < m0 ? k : m0 - 1;
            u[j] = static_cast<uint32_t>(src[kc]);
            v[j] = static_cast<uint32_t>(dst[kc]);
            tk[j] = ts_key(ts[kc]);
        }
#pragma unroll
        for (int j = 0; j < kEdgeUnroll; j++) {
            const int64_t k = k0 + static_cast<int64_t>(j) * kBlock;
            if (k >= m0) continue;
            keys[k] = make_key(L, u[j], tk[j], L.packed ? v[j] : 0u);
            vals[k] = static_cast<uint32_t>(k);
            if (both) {
                keys[m0 + k] = make_key(L, v[j], tk[j], L.packed ? u[j] : 0u);
                vals[m0 + k] = static_cast<uint32_t>(m0 + k);
            }
        }
    }
}

// Lanes of the wave whose (valid) BITS-bit digit equals this lane's digit.
template <int BITS>
__device__ __forceinline__ uint64_t match_digit(uint32_t d, bool valid) {
    uint64_t m = __ballot(valid);
#pragma unroll
    for (int b = 0; b < BITS; b++) {
        const bool bit = (d >> b) & 1u;
        const uint64_t bb = __ballot(bit);
        m &= bit ? bb : ~bb;
    }
    return m;
}

// Per-tile digit counts, stored digit-major: hist[d * ntiles + tile], for the
// 2^BITS digits (key >> shift) & (2^BITS - 1).
template <int BITS>
__global__ __launch_bounds__(kBlock) void radix_upsweep_kernel(const uint64_t *__restrict__ keys,
                                                               int64_t M, int shift,
                                                               uint32_t *__restrict__ hist,
                                                               int64_t ntiles) {
    constexpr int B = 1 << BITS;
    static_assert(B <= kBlock, "one thread per digit");
    __shared__ uint32_t cnt[B];
    const int64_t tile = radix_tile(ntiles);
    if (tile < 0) return;                           // block-uniform
    if (threadIdx.x < B) cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = tile * kTile;
    const uint64_t lane_bit = 1ull << lane_id();
    // every key of the tile is loaded before any is counted: the index is
    // clamped rather than the load predicated, so that the loads issue back to
    // back (a key past M is read from M - 1 and not counted)
    uint32_t dg[kTileItems];
#pragma unroll
    for (int r = 0; r < kTileItems; r++) {
        const int64_t idx = base + static_cast<int64_t>(r) * kBlock + threadIdx.x;
        dg[r] = static_cast<uint32_t>(keys[idx < M ? idx : M - 1] >> shift) & (B - 1);
    }
#pragma unroll
    for (int r = 0; r < kTileItems; r++) {
        const bool valid = base + static_cast<int64_t>(r) * kBlock + threadIdx.x < M;
        const uint64_t peers = match_digit<BITS>(dg[r], valid);
        if (valid && (peers & (lane_bit - 1)) == 0) atomicAdd(&cnt[dg[r]], static_cast<uint32_t>(__popcll(peers)));
    }
    __syncthreads();
    if (threadIdx.x < B) hist[static_cast<int64_t>(threadIdx.x) * ntiles + tile] = cnt[threadIdx.x];
}

// Stable scatter of one tile by its BITS-bit digit.  hist_off holds the
// exclusive scan of hist (digit-major), i.e. where this tile's keys of digit
// d start.
template <int BITS>
__global__ __launch_bounds__(kBlock) void radix_downsweep_kernel(
    const uint64_t *__restrict__ kin, const uint32_t *__restrict__ vin, uint64_t *__restrict__ kout,
    uint32_t *__restrict__ vout, int64_t M, int shift, const uint32_t *__restrict__ hist_off,
    int64_t ntiles) {
    constexpr int B = 1 << BITS;
    static_assert(B <= kBlock, "one thread per digit");
    __shared__ uint64_t sk[kTile];
    __shared__ uint32_t sv[kTile];
    __shared__ uint32_t wcnt[kWaves][B];
    __shared__ uint32_t bdo[B];
    __shared__ uint32_t gofs[B];
    __shared__ uint32_t scan_lds[kBlock / kWave];

    const int w = threadIdx.x / kWave;
    const int lane = lane_id();
    const uint64_t lane_bit = 1ull << lane;
    const int64_t tile = radix_tile(ntiles);
    if (tile < 0) return;                           // block-uniform
    if (threadIdx.x < B) {
#pragma unroll
        for (int i = 0; i < kWaves; i++) wcnt[i][threadIdx.x] = 0;
    }
    __syncthreads();

    const int64_t tile0 = tile * kTile;
    const int64_t base = tile0 + static_cast<int64_t>(w) * kWaveTile;
    uint64_t key[kTileItems];
    uint32_t val[kTileItems];
    uint32_t rank[kTileItems];
#pragma unroll
    for (int r = 0; r < kTileItems; r++) {
        const int64_t idx = base + static_cast<int64_t>(r) * kWave + lane;
        const bool valid = idx < M;
        key[r] = valid ? kin[idx] : ~0ull;
        val[r] = valid ? vin[idx] : 0u;
    }
#pragma unroll
    for (int r = 0; r < kTileItems; r++) {
        const int64_t idx = base + static_cast<int64_t>(r) * kWave + lane;
        const bool valid = idx < M;
        const uint32_t d = static_cast<uint32_t>(key[r] >> shift) & (B - 1);
        const uint64_t peers = match_digit<BITS>(d, valid);
        const uint64_t below = peers & (lane_bit - 1);
        const uint32_t prior = wcnt[w][d];
        rank[r] = prior + static_cast<uint32_t>(__popcll(below));
        if (valid && below == 0) wcnt[w][d] = prior + static_cast<uint32_t>(__popcll(peers));
        // the next round's reads must follow this round's update
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    __syncthreads();

    // per digit: exclusive bases across the waves, tile total, global offset
    {
        const int d = threadIdx.x;
        uint32_t run = 0;
        if (d < B) {
#pragma unroll
            for (int i = 0; i < kWaves; i++) {
                const uint32_t c = wcnt[i][d];
                wcnt[i][d] = run;
                run += c;
            }
            gofs[d] = hist_off[static_cast<int64_t>(d) * ntiles + tile];
        }
        uint32_t total;
        const uint32_t ex = block_exclusive_sum<uint32_t>(run, scan_lds, &total);   // every thread takes part
        if (d < B) bdo[d] = ex;
    }
    __syncthreads();

#pragma unroll
    for (int r = 0; r < kTileItems; r++) {
        const int64_t idx = base + static_cast<int64_t>(r) * kWave + lane;
        if (idx < M) {
            const uint32_t d = static_cast<uint32_t>(key[r] >> shift) & (B - 1);
            const uint32_t pos = bdo[d] + wcnt[w][d] + rank[r];
            sk[pos] = key[r];
            sv[pos] = val[r];
        }
    }
    __syncthreads();

    const int64_t left = M - tile0;
    const int n = left < kTile ? static_cast<int>(left) : kTile;
    for (int i = threadIdx.x; i < n; i += kBlock) {
        const uint64_t k = sk[i];
        const uint32_t d = static_cast<uint32_t>(k >> shift) & (B - 1);
        const int64_t g = static_cast<int64_t>(gofs[d]) + (i - static_cast<int64_t>(bdo[d]));
        if (g >= 0 && g < M) {     // always true for consistent counts; keeps stores in bounds
            kout[g] = k;
            vout[g] = sv[i];
        }
    }
}

// Each node's first timestamp as a value of type F that orders like it: the
// float itself, or (packed layout, F = uint8_t / uint16_t) the key's
// timestamp field, whose bits outside the field are the same in every entry.
template <class F>
__device__ __forceinline__ F first_value(const KeyLayout &L, uint64_t k) {
    if constexpr (sizeof(F) == sizeof(float)) {
        return key_ts(key_tskey(L, k));
    } else {
        return static_cast<F>((k >> L.nbr_bits) & low_mask(L.ts_bits));
    }
}

// A value above every first_value<F>, for nodes without entries: +inf, or all
// ones (not below any field value, which decides the hint as +inf does).
template <class F>
__host__ __device__ __forceinline__ F first_none() {
    if constexpr (sizeof(F) == sizeof(float)) {
        return __builtin_inff();
    } else {
        return static_cast<F>(~static_cast<F>(0));
    }
}

// Entries handled per lane by the wavefront-tiled kernels below: a wavefront
// takes kEmitPerLane * 64 consecutive sorted entries, lane l the entries
// base + l + 64 j, so every load and store of a round is coalesced and all of
// them are in flight together.
constexpr int kEmitPerLane = 4;
constexpr int kEmitSpan = kEmitPerLane * kWave;

// 64-bit lane shuffle (two 32-bit halves).
__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src) {
    const uint32_t lo = static_cast<uint32_t>(__shfl(static_cast<int>(static_cast<uint32_t>(v)), src, kWave));
    const uint32_t hi = static_cast<uint32_t>(__shfl(static_cast<int>(static_cast<uint32_t>(v >> 32)), src, kWave));
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Sorted keys base + l + 64 j (j < kEmitPerLane) and the key before each:
// the lane below, lane 63 of the previous round, or keys[base - 1].  Entries
// at or past M get the last key; callers skip them.
__device__ __forceinline__ void load_keys_prev(const uint64_t *__restrict__ keys, int64_t M, int64_t base, int lane,
                                               uint64_t (&key)[kEmitPerLane], uint64_t (&prev)[kEmitPerLane]) {
#pragma unroll
    for (int j = 0; j < kEmitPerLane; j++) {
        const int64_t p = base + j * kWave + lane;
        // clamped, not predicated, so that the loads issue together: a lane past
        // the end holds the last key, and its caller skips it
        key[j] = keys[p < M ? p : M - 1];
    }
    const uint64_t before = base > 0 ? keys[base - 1] : ~0ull;   // same address in every lane
#pragma unroll
    for (int j = 0; j < kEmitPerLane; j++) {
        const uint64_t below = shfl64(key[j], lane == 0 ? 0 : lane - 1);
        const uint64_t wrap = j > 0 ? shfl64(key[j - 1], kWave - 1) : before;
        prev[j] = lane == 0 ? wrap : below;
    }
}

// first[x] = first_value of node x's first entry in the sorted keys (the
// caller fills first with first_none beforehand, for nodes without entries).
template <class F>
__global__ __launch_bounds__(kBlock) void first_ts_kernel(const uint64_t *__restrict__ keys, int64_t M,
                                                          const KeyLayout L, F *__restrict__ first) {
    const int lane = lane_id();
    const int64_t wave = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) / kWave;
    const int64_t waves = static_cast<int64_t>(gridDim.x) * (kBlock / kWave);
    for (int64_t base = wave * kEmitSpan; base < M; base += waves * kEmitSpan) {
        uint64_t key[kEmitPerLane], prev[kEmitPerLane];
        load_keys_prev(keys, M, base, lane, key, prev);
#pragma unroll
        for (int j = 0; j < kEmitPerLane; j++) {
            const int64_t p = base + j * kWave + lane;
            const uint32_t u = key_node(L, key[j]);
            if (p < M && (p == 0 || key_node(L, prev[j]) != u)) first[u] = first_value<F>(L, key[j]);
        }
    }
}

template <class F>
__global__ __launch_bounds__(kBlock) void fill_first_kernel(F *__restrict__ a, int64_t n) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n; i += stride)
        a[i] = first_none<F>();
}

// Writes entries[p] from the sorted (key, i) and fills indptr: node x starts
// at the first p whose owner is >= x.  The neighbour comes from the key
// (packed layout) or from the edge list; with `first` (each node's
// first_value) the entry's TGL_NBR_FIRST hint is set here.  Wavefront-tiled
// like first_ts_kernel: each lane's gathers (neighbour, eid, first value) for
// its kEmitPerLane entries are issued together.
template <class F>
__global__ __launch_bounds__(kBlock) void emit_kernel(const uint64_t *__restrict__ keys,
                                                      const uint32_t *__restrict__ vals, int64_t M,
                                                      int64_t m0, const int32_t *__restrict__ src,
                                                      const int32_t *__restrict__ dst,
                                                      const int64_t *__restrict__ eid, int64_t N,
                                                      const KeyLayout L, const F *__restrict__ first,
                                                      int64_t *__restrict__ indptr,
                                                      int4 *__restrict__ ent,
                                                      float *__restrict__ ts_out) {
    const int lane = lane_id();
    const int64_t wave = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) / kWave;
    const int64_t waves = static_cast<int64_t>(gridDim.x) * (kBlock / kWave);
    for (int64_t base = wave * kEmitSpan; base < M; base += waves * kEmitSpan) {
        uint64_t key[kEmitPerLane], prev[kEmitPerLane];
        int64_t k[kEmitPerLane];
        bool fwd[kEmitPerLane];
#pragma unroll
        for (int j = 0; j < kEmitPerLane; j++) {
            const int64_t p = base + j * kWave + lane;
            int64_t i = static_cast<int64_t>(vals[p < M ? p : M - 1]);   // past the end: the last entry's
            if (i >= M) i = 0;   // never taken for a permutation; keeps loads in bounds
            fwd[j] = i < m0;
            k[j] = fwd[j] ? i : i - m0;
        }
        load_keys_prev(keys, M, base, lane, key, prev);
        int32_t v[kEmitPerLane];
        int64_t e[kEmitPerLane];
#pragma unroll
        for (int j = 0; j < kEmitPerLane; j++) {
            v[j] = L.packed ? static_cast<int32_t>(key[j] & low_mask(L.nbr_bits)) : (fwd[j] ? dst[k[j]] : src[k[j]]);
            e[j] = eid ? eid[k[j]] : k[j];
        }
        bool hint[kEmitPerLane];
#pragma unroll
        for (int j = 0; j < kEmitPerLane; j++)
            hint[j] = first && v[j] >= 0 && v[j] < N && !(first[v[j]] < first_value<F>(L, key[j]));
#pragma unroll
        for (int j = 0; j < kEmitPerLane; j++) {
            const int64_t p = base + j * kWave + lane;
            if (p >= M) continue;
            const int64_t u = static_cast<int64_t>(key_node(L, key[j]));
            const float t = key_ts(key_tskey(L, key[j]));
            const uint32_t vw = static_cast<uint32_t>(v[j]) | (hint[j] ? TGL_NBR_FIRST : 0u);
            ent[p] = make_int4(static_cast<int>(vw), __float_as_int(t), static_cast<int>(static_cast<uint32_t>(e[j])),
                               static_cast<int>(static_cast<uint64_t>(e[j]) >> 32));
            ts_out[p] = t;
            // owners are in [0, N) after validation; the clamps only bound the stores
            const int64_t uprev = p == 0 ? -1 : static_cast<int64_t>(key_node(L, prev[j]));
            const int64_t x1 = u < N ? u : N - 1;
            for (int64_t x = uprev + 1; x <= x1; x++) indptr[x] = p;
            if (p == M - 1)
                for (int64_t x = x1 + 1; x <= N; x++) indptr[x] = M;
        }
    }
}

// Per-node records {start, end, first ts, last ts, ts[0..27]}: eight lanes per
// node, lane i writing the i-th 16 bytes of the node's 128-byte record.  If
// first_out is given, the first timestamps also go to first_out[x].
__global__ __launch_bounds__(kBlock) void nodes_kernel(const int64_t *__restrict__ indptr,
                                                       const float *__restrict__ ts, int64_t N, int64_t M,
                                                       int4 *__restrict__ nodes, float *__restrict__ first_out) {
    constexpr int kParts = static_cast<int>(sizeof(tgl_node) / 16);
    static_assert(sizeof(tgl_node) == 128 && TGL_NODE_INLINE == 4 * (kParts - 1), "node record layout");
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    const int64_t total = N * kParts;
    for (int64_t g = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; g < total; g += stride) {
        const int64_t x = g / kParts;
        const int part = static_cast<int>(g - x * kParts);
        int64_t a = indptr[x];
        int64_t b = indptr[x + 1];
        a = a < 0 ? 0 : (a > M ? M : a);
        b = b < a ? a : (b > M ? M : b);
        int4 v;
        if (part == 0) {
            const float first = b > a ? ts[a] : __builtin_inff();
            const float last = b > a ? ts[b - 1] : -__builtin_inff();
            v = make_int4(static_cast<int>(static_cast<uint32_t>(a)), static_cast<int>(static_cast<uint32_t>(b)),
                          __float_as_int(first), __float_as_int(last));
            if (first_out) first_out[x] = first;
        } else {
            const int64_t p = a + 4 * (part - 1);
            const float inf = __builtin_inff();
            v = make_int4(__float_as_int(p < b ? ts[p] : inf), __float_as_int(p + 1 < b ? ts[p + 1] : inf),
                          __float_as_int(p + 2 < b ? ts[p + 2] : inf), __float_as_int(p + 3 < b ? ts[p + 3] : inf));
        }
        nodes[g] = v;
    }
}

// TGL_NBR_FIRST hints: bit 31 of entry p's neighbour id is set exactly when
// the neighbour's first timestamp is not below ts[p] (its run is sorted, so
// no entry of it lies below ts[p]).  first[x * stride] is node x's first
// timestamp (+inf for an empty run): a compact array (stride 1) or the node
// records (stride 32, offset to the first_ts word by the caller).  Neighbour
// ids outside [0, N) get a clear bit.
__global__ __launch_bounds__(kBlock) void first_hint_kernel(int4 *__restrict__ ent, const float *__restrict__ ts,
                                                            int64_t M, const float *__restrict__ first,
                                                            int64_t stride, int64_t N) {
    int32_t *const nb = reinterpret_cast<int32_t *>(ent);         // word 0 of every 16-byte entry
    const int64_t gstride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t p = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; p < M; p += gstride) {
        const uint32_t raw = static_cast<uint32_t>(nb[4 * p]);
        const uint32_t x = raw & TGL_NBR_MASK;
        bool hint = false;
        if (static_cast<int64_t>(x) < N) hint = !(first[static_cast<int64_t>(x) * stride] < ts[p]);
        const uint32_t out = x | (hint ? TGL_NBR_FIRST : 0u);
        if (out != raw) nb[4 * p] = static_cast<int32_t>(out);
    }
}

// Neighbour histories (tgl_span): entry p with neighbour v and time t gets
// hist[p] = {lo, hi}, lo the start of v's run and hi = lo + #{entries of v
// with ts < t} -- where a root (v, t) of a later hop finds its candidates
// when windows are unbounded below.  v's node record answers alone when t is
// at or below its first timestamp, above its last, or inside the first
// TGL_NODE_INLINE timestamps (held in the record); otherwise a binary search
// of the rest of the run, which then holds an entry at or above t (the last
// one).  A neighbour id outside [0, N) gets {0, 0}.  With set_hint, the
// entry's TGL_NBR_FIRST bit is written from the span (hi == lo: no entry of
// v below t) over a clear bit.  Wavefront-tiled like emit_kernel, so that
// each lane's record loads for its kEmitPerLane entries are in flight
// together.
__global__ __launch_bounds__(kBlock) void hist_kernel(int4 *__restrict__ ent, const float *__restrict__ ts,
                                                      int64_t M, const int4 *__restrict__ nodes, int64_t N,
                                                      uint2 *__restrict__ hist, bool set_hint) {
    int2 *const head = reinterpret_cast<int2 *>(ent);        // (nbr, ts) of each 16-byte entry
    const uint32_t um = static_cast<uint32_t>(M);
    const int lane = lane_id();
    const int64_t wave = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) / kWave;
    const int64_t waves = static_cast<int64_t>(gridDim.x) * (kBlock / kWave);
    for (int64_t base = wave * kEmitSpan; base < M; base += waves * kEmitSpan) {
        int2 e[kEmitPerLane];
#pragma unroll
        for (int j = 0; j < kEmitPerLane; j++) {
            const int64_t p = base + j * kWave + lane;
            e[j] = head[2 * (p < M ? p : M - 1)];
        }
        int4 h[kEmitPerLane];
#pragma unroll
        for (int j = 0; j < kEmitPerLane; j++) {
            const uint32_t x = static_cast<uint32_t>(e[j].x) & TGL_NBR_MASK;
            h[j] = nodes[static_cast<int64_t>(static_cast<int64_t>(x) < N ? x : 0u) * 8];   // record 0 stands in
        }
#pragma unroll
        for (int j = 0; j < kEmitPerLane; j++) {
            const int64_t p = base + j * kWave + lane;
            if (p >= M) continue;
            const uint32_t x = static_cast<uint32_t>(e[j].x) & TGL_NBR_MASK;
            const float t = __int_as_float(e[j].y);
            uint32_t lo = 0, hi = 0;
            if (static_cast<int64_t>(x) < N) {
                uint32_t a = static_cast<uint32_t>(h[j].x), b = static_cast<uint32_t>(h[j].y);
                a = a > um ? um : a;
                b = b < a ? a : (b > um ? um : b);
                lo = a;
                if (!(__int_as_float(h[j].z) < t)) {
                    hi = a;                               // nothing below t (or t is NaN)
                } else if (__int_as_float(h[j].w) < t) {
                    hi = b;                               // the whole run
                } else {
                    const int4 *const rec = nodes + static_cast<int64_t>(x) * 8;
                    uint32_t c = 0;                       // inline timestamps below t (+inf past the run)
#pragma unroll
                    for (int q = 1; q <= TGL_NODE_INLINE / 4; q++) {
                        const int4 w = rec[q];
                        c += (__int_as_float(w.x) < t) + (__int_as_float(w.y) < t) + (__int_as_float(w.z) < t) +
                             (__int_as_float(w.w) < t);
                    }
                    if (c < TGL_NODE_INLINE || b - a <= TGL_NODE_INLINE) {
                        hi = a + c;
                    } else {
                        // the first position of [a + TGL_NODE_INLINE, b) with ts >= t;
                        // ts[b - 1] (the last timestamp) is one
                        uint32_t l = a + TGL_NODE_INLINE, r = b - 1;
                        while (l < r) {
                            const uint32_t m = l + (r - l) / 2;
                            if (ts[m] < t) l = m + 1;
                            else r = m;
                        }
                        hi = l;
                    }
                }
                if (set_hint && hi == lo) head[2 * p].x = static_cast<int>(x | TGL_NBR_FIRST);
            }
            hist[p] = make_uint2(lo, hi);
        }
    }
}

// Search index: every TGL_INDEX_STRIDE-th timestamp.
__global__ __launch_bounds__(kBlock) void index_kernel(const float *__restrict__ ts, int64_t L,
                                                       float *__restrict__ idx) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; j < L; j += stride)
        idx[j] = ts[j * TGL_INDEX_STRIDE];
}

// Time directory (tgl_cell), one lane per search-index slot j: the node x
// whose run [a, b) holds entry p = j * TGL_INDEX_STRIDE (the last x with
// indptr[x] <= p, by a binary search of indptr), then the first position of
// the run whose timestamp falls in cell k = j - ceil(a / TGL_INDEX_STRIDE)
// or later, or b if there is none (a binary search of the run on the cells
// of its timestamps; a run whose timestamps are all equal has every entry
// in cell 0).  The run bounds and first and last timestamps come from the
// node records, which the sampler reads too.  A slot whose entry the
// record's run does not hold (only with a malformed indptr) gets {a, +inf}.
__global__ __launch_bounds__(kBlock) void dir_kernel(const int64_t *__restrict__ indptr,
                                                     const float *__restrict__ ts, const int4 *__restrict__ nodes,
                                                     int64_t N, int64_t M, int64_t L, uint2 *__restrict__ dir) {
    constexpr uint32_t X = TGL_INDEX_STRIDE;
    const uint32_t um = static_cast<uint32_t>(M);
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; j < L; j += stride) {
        const int64_t p = j * X;
        int64_t lo = 0, hi = N - 1;
        while (lo < hi) {
            const int64_t mid = lo + (hi - lo + 1) / 2;
            if (indptr[mid] <= p) lo = mid;
            else hi = mid - 1;
        }
        const int4 r = nodes[lo * 8];
        uint32_t a = static_cast<uint32_t>(r.x), b = static_cast<uint32_t>(r.y);
        a = a > um ? um : a;
        b = b < a ? a : (b > um ? um : b);
        uint32_t pos = a;
        float cts = __builtin_inff();
        if (p >= a && p < b) {
            const float f = __int_as_float(r.z), l = __int_as_float(r.w);
            const uint32_t ja = a / X + (a % X != 0);
            const uint32_t K = b / X + (b % X != 0) - ja;
            const uint32_t k = static_cast<uint32_t>(j) - ja;
            if (k > 0) {
                const float sc = dir_scale(f, l, K);
                uint32_t l2 = a, r2 = b;
                while (l2 < r2) {
                    const uint32_t m = l2 + (r2 - l2) / 2;
                    if (dir_cell(ts[m], f, l, sc, K) < k) l2 = m + 1;
                    else r2 = m;
                }
                pos = l2;
            }
            if (pos < b) cts = ts[pos];
        }
        dir[j] = make_uint2(pos, __float_as_uint(cts));
    }
}

// Columns to 16-byte entries: entry p = {nbr[p] with bit 31 clear, ts[p],
// eid[p] (p when eid is null)}.
__global__ __launch_bounds__(kBlock) void pack_kernel(const int32_t *__restrict__ nbr, const float *__restrict__ ts,
                                                      const int64_t *__restrict__ eid, int64_t M,
                                                      int4 *__restrict__ ent) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t p = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; p < M; p += stride) {
        const int64_t e = eid ? eid[p] : p;
        ent[p] = make_int4(static_cast<int>(static_cast<uint32_t>(nbr[p]) & TGL_NBR_MASK), __float_as_int(ts[p]),
                           static_cast<int>(static_cast<uint32_t>(e)),
                           static_cast<int>(static_cast<uint32_t>(static_cast<uint64_t>(e) >> 32)));
    }
}

// 16-byte entries to columns: nbr (bit 31 cleared) and eid, each optional.
__global__ __launch_bounds__(kBlock) void unpack_kernel(const int4 *__restrict__ ent, int64_t M,
                                                        int32_t *__restrict__ nbr, int64_t *__restrict__ eid) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t p = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; p < M; p += stride) {
        const int4 v = ent[p];
        if (nbr) nbr[p] = static_cast<int32_t>(static_cast<uint32_t>(v.x) & TGL_NBR_MASK);
        if (eid) eid[p] = static_cast<int64_t>(static_cast<uint32_t>(v.z)) | (static_cast<int64_t>(v.w) << 32);
    }
}

__global__ __launch_bounds__(kBlock) void fill_indptr_kernel(int64_t *__restrict__ indptr, int64_t n,
                                                             int64_t value) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n; i += stride)
        indptr[i] = value;
}

struct BuildWs {
    BuildFlags *flags = nullptr;
    uint64_t *keys[2] = {nullptr, nullptr};
    uint32_t *vals[2] = {nullptr, nullptr};
    uint32_t *hist = nullptr;
    int64_t *partials = nullptr;
    int64_t ntiles = 0;
    size_t bytes = 0;
};

BuildWs carve_build_ws(void *base, int64_t M) {
    BuildWs w;
    Carver cv(base);
    w.ntiles = (M + kTile - 1) / kTile;
    w.flags = cv.take<BuildFlags>(1);
    for (int i = 0; i < 2; i++) {
        w.keys[i] = cv.take<uint64_t>(static_cast<size_t>(M));
        w.vals[i] = cv.take<uint32_t>(static_cast<size_t>(M));
    }
    const int64_t nh = w.ntiles * kBins;
    w.hist = cv.take<uint32_t>(static_cast<size_t>(nh));
    w.partials = cv.take<int64_t>(static_cast<size_t>(scan_tiles(nh) + 1));
    w.bytes = cv.size();
    return w;
}

bool build_args_ok(int64_t num_edges, int64_t num_nodes, uint32_t flags) {
    if (num_edges < 0 || num_nodes < 1 || num_nodes > INT32_MAX) return false;
    if (flags & ~TGL_BUILD_UNDIRECTED) return false;
    const int64_t M = (flags & TGL_BUILD_UNDIRECTED) ? 2 * num_edges : num_edges;
    return M <= kMaxEntries && num_edges <= kMaxEntries;
}

// Lowest varying bit and number of bits from it to the highest varying bit.
void field_of(uint32_t varying, int *lo, int *bits) {
    if (varying == 0) {
        *lo = 0;
        *bits = 0;
        return;
    }
    *lo = __builtin_ctz(varying);
    *bits = 32 - __builtin_clz(varying) - *lo;
}

// The packed layout when node field, tskey field and neighbour id fit in 64
// bits, else the plain one.  Neighbour ids take the bits of N - 1.
KeyLayout key_layout(const BuildFlags &f, int64_t N) {
    KeyLayout L{};
    const uint32_t node_or = static_cast<uint32_t>(f.or_bits >> 32), node_and = static_cast<uint32_t>(f.and_bits >> 32);
    const uint32_t ts_or = static_cast<uint32_t>(f.or_bits), ts_and = static_cast<uint32_t>(f.and_bits);
    field_of(node_or ^ node_and, &L.node_lo, &L.node_bits);
    field_of(ts_or ^ ts_and, &L.ts_lo, &L.ts_bits);
    const uint32_t top = static_cast<uint32_t>(N - 1);
    L.nbr_bits = top == 0 ? 0 : 32 - __builtin_clz(top);
    L.node_konst = node_and & ~static_cast<uint32_t>(low_mask(L.node_bits) << L.node_lo);
    L.ts_konst = ts_and & ~static_cast<uint32_t>(low_mask(L.ts_bits) << L.ts_lo);
    L.packed = L.node_bits + L.ts_bits + L.nbr_bits <= 64;
    return L;
}

// Key bits the sort must order by: the varying node and tskey bits where the
// layout puts them (never the neighbour bits, so ties keep input order).
uint64_t sort_bits(const KeyLayout &L, const BuildFlags &f) {
    const uint64_t var = f.or_bits ^ f.and_bits;
    if (!L.packed) return var;
    const uint64_t nv = ((var >> 32) >> L.node_lo) & low_mask(L.node_bits);
    const uint64_t tv = ((var & 0xFFFFFFFFull) >> L.ts_lo) & low_mask(L.ts_bits);
    const int node_at = L.nbr_bits + L.ts_bits;
    return (node_at < 64 ? nv << node_at : 0ull) | (tv << L.nbr_bits);
}

unsigned grid_for(int64_t n, int64_t cap = 1 << 16) {
    int64_t b = (n + kBlock - 1) / kBlock;
    if (b < 1) b = 1;
    if (b > cap) b = cap;
    return static_cast<unsigned>(b);
}

}  // namespace
}  // namespace tgl

using namespace tgl;

extern "C" {

size_t tgl_tcsr_build_workspace(int64_t num_edges, int64_t num_nodes, uint32_t flags) {
    if (!build_args_ok(num_edges, num_nodes, flags)) return 0;
    const int64_t M = (flags & TGL_BUILD_UNDIRECTED) ? 2 * num_edges : num_edges;
    return carve_build_ws(nullptr, M).bytes;
}

tgl_status tgl_tcsr_build(const int32_t *src, const int32_t *dst, const float *ts,
                          const int64_t *eid, int64_t num_edges, int64_t num_nodes,
                          uint32_t flags, int64_t *indptr, tgl_entry *entries, float *ts_out,
                          tgl_node *nodes_out, float *ts_index_out, tgl_span *hist_out,
                          tgl_cell *dir_out, void *workspace, size_t workspace_bytes, void *stream) {
    if (!build_args_ok(num_edges, num_nodes, flags)) return TGL_EINVAL;
    if (num_edges > 0 && (!src || !dst || !ts || !entries || !ts_out)) return TGL_EINVAL;
    if (!indptr || !nodes_out) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(nodes_out) & 127u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(ts_index_out) & 15u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(hist_out) & 7u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(dir_out) & 7u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(entries) & 15u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(ts_out) & 15u) != 0) return TGL_EINVAL;
    const int64_t m0 = num_edges;
    const int64_t M = (flags & TGL_BUILD_UNDIRECTED) ? 2 * m0 : m0;
    const BuildWs need = carve_build_ws(nullptr, M);
    if (!workspace || workspace_bytes < need.bytes) return TGL_ENOSPACE;
    const BuildWs w = carve_build_ws(workspace, M);
    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    ScopedTimer tm(TGL_TIMER_BUILD, st);

    if (M == 0) {
        fill_indptr_kernel<<<grid_for(num_nodes + 1), kBlock, 0, st>>>(indptr, num_nodes + 1, 0);
        nodes_kernel<<<grid_for(num_nodes * 8), kBlock, 0, st>>>(indptr, ts_out, num_nodes, 0,
                                                                 reinterpret_cast<int4 *>(nodes_out), nullptr);
        return launch_status();
    }

    init_flags_kernel<<<1, 1, 0, st>>>(w.flags);
    const unsigned ge = grid_for((m0 + kEdgeUnroll - 1) / kEdgeUnroll);
    reduce_kernel<<<ge, kBlock, 0, st>>>(src, dst, ts, m0, M != m0, num_nodes, w.flags);
    if (launch_status() != TGL_OK) return TGL_EDEVICE;
    BuildFlags hf{};
    if (hipMemcpyAsync(&hf, w.flags, sizeof(hf), hipMemcpyDeviceToHost, st) != hipSuccess)
        return TGL_EDEVICE;
    if (hipStreamSynchronize(st) != hipSuccess) return TGL_EDEVICE;
    if (hf.err) return TGL_ERANGE;

    const KeyLayout L = key_layout(hf, num_nodes);
    const uint64_t varying = sort_bits(L, hf);
    keys_kernel<<<ge, kBlock, 0, st>>>(src, dst, ts, m0, M != m0, L, w.keys[0], w.vals[0]);
    int cur = 0;
    // Digits from the lowest varying sort bit up (in the packed layout the
    // neighbour bits lie below every sort bit: they must not take part, or
    // ties would leave input order).  The span from there to the highest
    // varying bit is cut into as few passes as 8-bit digits allow, `step`
    // bits apart (c4: 35 bits, five 7-bit digits).  A pass reads a digit of
    // kb = 7 or 8 bits at its shift; when step is below 7 the digits overlap,
    // which leaves the LSD order unchanged.  A digit on which every key agrees
    // is skipped.
    const int lo_bit = varying == 0 ? 0 : __builtin_ctzll(varying);   // packed: never below the neighbour bits
    const int hi_bit = varying == 0 ? lo_bit : 64 - __builtin_clzll(varying);
    const int span = hi_bit > lo_bit ? hi_bit - lo_bit : 0;
    const int npass = (span + kMaxRadixBits - 1) / kMaxRadixBits;
    const int step = npass > 0 ? (span + npass - 1) / npass : kMaxRadixBits;
    const int kb = step == 8 ? 8 : 7;
    const int64_t nh = w.ntiles << kb;
    const int64_t sc_tiles = scan_tiles(nh);
    for (int pass = 0; pass < npass; pass++) {
        const int shift = lo_bit + pass * step;
        if (((varying >> shift) & ((uint64_t(1) << kb) - 1)) == 0) continue;   // every key has this digit
        if (kb == 8)
            radix_upsweep_kernel<8><<<radix_grid(w.ntiles), kBlock, 0, st>>>(w.keys[cur], M, shift, w.hist,
                                                                                       w.ntiles);
        else
            radix_upsweep_kernel<7><<<radix_grid(w.ntiles), kBlock, 0, st>>>(w.keys[cur], M, shift, w.hist,
                                                                                       w.ntiles);
        scan_reduce_kernel<uint32_t><<<static_cast<unsigned>(sc_tiles), kBlock, 0, st>>>(
            w.hist, nh, nullptr, w.partials);
        launch_scan_partials(w.partials, sc_tiles, nullptr, st);
        scan_apply_kernel<uint32_t, uint32_t><<<static_cast<unsigned>(sc_tiles), kBlock, 0, st>>>(
            w.hist, w.hist, nh, nullptr, w.partials);
        if (kb == 8)
            radix_downsweep_kernel<8><<<radix_grid(w.ntiles), kBlock, 0, st>>>(
                w.keys[cur], w.vals[cur], w.keys[cur ^ 1], w.vals[cur ^ 1], M, shift, w.hist, w.ntiles);
        else
            radix_downsweep_kernel<7><<<radix_grid(w.ntiles), kBlock, 0, st>>>(
                w.keys[cur], w.vals[cur], w.keys[cur ^ 1], w.vals[cur ^ 1], M, shift, w.hist, w.ntiles);
        if (launch_status() != TGL_OK) return TGL_EDEVICE;
        cur ^= 1;
    }
    // Each node's first timestamp, read from the sorted keys into the sort's
    // spare key buffer (8 bytes per entry) when it fits, so that the entries
    // are written with their neighbour-first hints; otherwise the hints are
    // set afterwards from the node records.
    // A packed timestamp field of at most 16 bits stands in for the float, so
    // that the neighbours' values are gathered from a smaller array.
    // With neighbour histories the hints come from them instead (an empty
    // history is the hint), and no first timestamps are needed.
    const int fbytes = L.packed && L.ts_bits <= 8 ? 1 : (L.packed && L.ts_bits <= 16 ? 2 : 4);
    void *const first = !hist_out && num_nodes * fbytes <= 8 * M ? static_cast<void *>(w.keys[cur ^ 1]) : nullptr;
    const unsigned gm = grid_for(M), gn = grid_for(num_nodes);
    int4 *const ent = reinterpret_cast<int4 *>(entries);
    if (first && fbytes == 1) {
        uint8_t *const f = static_cast<uint8_t *>(first);
        fill_first_kernel<uint8_t><<<gn, kBlock, 0, st>>>(f, num_nodes);
        first_ts_kernel<uint8_t><<<gm, kBlock, 0, st>>>(w.keys[cur], M, L, f);
        emit_kernel<uint8_t><<<gm, kBlock, 0, st>>>(w.keys[cur], w.vals[cur], M, m0, src, dst, eid, num_nodes, L, f,
                                                    indptr, ent, ts_out);
    } else if (first && fbytes == 2) {
        uint16_t *const f = static_cast<uint16_t *>(first);
        fill_first_kernel<uint16_t><<<gn, kBlock, 0, st>>>(f, num_nodes);
        first_ts_kernel<uint16_t><<<gm, kBlock, 0, st>>>(w.keys[cur], M, L, f);
        emit_kernel<uint16_t><<<gm, kBlock, 0, st>>>(w.keys[cur], w.vals[cur], M, m0, src, dst, eid, num_nodes, L,
                                                     f, indptr, ent, ts_out);
    } else {
        float *const f = static_cast<float *>(first);
        if (f) {
            fill_first_kernel<float><<<gn, kBlock, 0, st>>>(f, num_nodes);
            first_ts_kernel<float><<<gm, kBlock, 0, st>>>(w.keys[cur], M, L, f);
        }
        emit_kernel<float><<<gm, kBlock, 0, st>>>(w.keys[cur], w.vals[cur], M, m0, src, dst, eid, num_nodes, L, f,
                                                  indptr, ent, ts_out);
    }
    nodes_kernel<<<grid_for(num_nodes * 8), kBlock, 0, st>>>(indptr, ts_out, num_nodes, M,
                                                             reinterpret_cast<int4 *>(nodes_out), nullptr);
    if (!first && !hist_out)
        first_hint_kernel<<<grid_for(M), kBlock, 0, st>>>(reinterpret_cast<int4 *>(entries), ts_out, M,
                                                          reinterpret_cast<const float *>(nodes_out) + 2, 32,
                                                          num_nodes);
    if (ts_index_out && M > 0) {
        const int64_t L = tgl_index_len(M);
        index_kernel<<<grid_for(L), kBlock, 0, st>>>(ts_out, L, ts_index_out);
    }
    if (hist_out)
        hist_kernel<<<grid_for((M + kEmitPerLane - 1) / kEmitPerLane), kBlock, 0, st>>>(
            reinterpret_cast<int4 *>(entries), ts_out, M, reinterpret_cast<const int4 *>(nodes_out), num_nodes,
            reinterpret_cast<uint2 *>(hist_out), true);
    if (dir_out) {
        const int64_t L = tgl_index_len(M);
        dir_kernel<<<grid_for(L), kBlock, 0, st>>>(indptr, ts_out, reinterpret_cast<const int4 *>(nodes_out),
                                                   num_nodes, M, L, reinterpret_cast<uint2 *>(dir_out));
    }
    return launch_status();
}

int64_t tgl_index_len(int64_t num_entries) {
    if (num_entries < 0) return -1;
    return num_entries / TGL_INDEX_STRIDE + (num_entries % TGL_INDEX_STRIDE != 0);
}

tgl_status tgl_tcsr_nodes(const int64_t *indptr, const float *ts, int64_t num_nodes,
                          int64_t num_entries, tgl_node *nodes, float *ts_index, tgl_entry *entries,
                          tgl_span *hist, tgl_cell *dir, void *stream) {
    if (num_nodes < 1 || num_nodes > INT32_MAX) return TGL_EINVAL;
    if (num_entries < 0 || num_entries > kMaxEntries) return TGL_EINVAL;
    if (!indptr || !nodes || (num_entries > 0 && !ts)) return TGL_EINVAL;
    if (hist && num_entries > 0 && !entries) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(nodes) & 127u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(ts_index) & 15u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(entries) & 15u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(hist) & 7u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(dir) & 7u) != 0) return TGL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    nodes_kernel<<<grid_for(num_nodes * 8), kBlock, 0, st>>>(indptr, ts, num_nodes, num_entries,
                                                             reinterpret_cast<int4 *>(nodes), nullptr);
    if (entries && num_entries > 0)
        first_hint_kernel<<<grid_for(num_entries), kBlock, 0, st>>>(
            reinterpret_cast<int4 *>(entries), ts, num_entries, reinterpret_cast<const float *>(nodes) + 2, 32,
            num_nodes);
    if (ts_index && num_entries > 0) {
        const int64_t L = tgl_index_len(num_entries);
        index_kernel<<<grid_for(L), kBlock, 0, st>>>(ts, L, ts_index);
    }
    if (hist && num_entries > 0)
        hist_kernel<<<grid_for((num_entries + kEmitPerLane - 1) / kEmitPerLane), kBlock, 0, st>>>(
            reinterpret_cast<int4 *>(entries), ts, num_entries, reinterpret_cast<const int4 *>(nodes), num_nodes,
            reinterpret_cast<uint2 *>(hist), false);
    if (dir && num_entries > 0) {
        const int64_t L = tgl_index_len(num_entries);
        dir_kernel<<<grid_for(L), kBlock, 0, st>>>(indptr, ts, reinterpret_cast<const int4 *>(nodes), num_nodes,
                                                   num_entries, L, reinterpret_cast<uint2 *>(dir));
    }
    return launch_status();
}

tgl_status tgl_tcsr_pack(const int32_t *nbr, const float *ts, const int64_t *eid, int64_t num_entries,
                         tgl_entry *entries, void *stream) {
    if (num_entries < 0 || num_entries > kMaxEntries) return TGL_EINVAL;
    if (num_entries > 0 && (!nbr || !ts || !entries)) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(entries) & 15u) != 0) return TGL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    if (num_entries > 0)
        pack_kernel<<<grid_for(num_entries), kBlock, 0, st>>>(nbr, ts, eid, num_entries,
                                                               reinterpret_cast<int4 *>(entries));
    return launch_status();
}

tgl_status tgl_tcsr_unpack(const tgl_entry *entries, int64_t num_entries, int32_t *nbr, int64_t *eid,
                           void *stream) {
    if (num_entries < 0 || num_entries > kMaxEntries) return TGL_EINVAL;
    if (num_entries > 0 && !entries) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(entries) & 15u) != 0) return TGL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    if (num_entries > 0 && (nbr || eid))
        unpack_kernel<<<grid_for(num_entries), kBlock, 0, st>>>(reinterpret_cast<const int4 *>(entries),
                                                                 num_entries, nbr, eid);
    return launch_status();
}

}  // extern "C"
