// tgl_gather.hip -- lookup of per-node and per-edge rows for sampled slots
// (Figure 2 of TGL, steps 2 and 3: node features, node memory and mailbox rows
// by neighbour id, edge features by edge id; Table 3 gives the row widths of
// the paper's datasets: 172-dim edge features on Wikipedia, 413 / 186 on
// GDELT, 768-dim node features on MAG).
//
// Every (slot, table) pair is an independent row copy, so the kernel is a
// plain HBM-bound gather: one wavefront copies kRows rows at a time, lane l
// moving 16-byte words l, l + 64, ... of each row.  The row keys are
// wavefront-uniform (one load by kRows lanes, then broadcast); the loads of
// all kRows rows are issued before any store, so a wavefront keeps kRows x
// 1 KB in flight per pass; outputs are written with nontemporal stores (they
// are consumed by the next stage, not re-read here).
#include "tgl_internal.hpp"

namespace tgl {
namespace {

using i32x4 = int __attribute__((ext_vector_type(4)));

constexpr int kRows = 8;   // rows per wavefront whose loads are in flight together

struct GatherTable {
    const i32x4 *rows;
    i32x4 *out;
    int64_t num_rows;
    int32_t words;         // 16-byte words per row
    int32_t key;           // TGL_KEY_NODE / TGL_KEY_EDGE
};

struct GatherArgs {
    const int32_t *nbr;
    const int64_t *eid;
    int64_t n;
    const int64_t *count;  // or null
    int64_t per;
    GatherTable t[TGL_MAX_TABLES];
    int32_t nt;
};

__global__ __launch_bounds__(kBlock) void gather_kernel(const GatherArgs a) {
    const int lane = lane_id();
    constexpr int kWaves = kBlock / kWave;
    const int64_t waves = static_cast<int64_t>(gridDim.x) * kWaves;
    const int64_t wave = __builtin_amdgcn_readfirstlane(static_cast<int>(blockIdx.x * kWaves + threadIdx.x / kWave));
    int64_t n = a.n;
    if (a.count) {
        // valid prefix: min(n, count * per), without overflowing the product
        const int64_t c = *a.count;
        const int64_t lim = c <= 0 ? 0 : (c > n / a.per ? n : c * a.per);
        n = lim < n ? lim : n;
    }
    const i32x4 zero = {0, 0, 0, 0};
    for (int ti = 0; ti < a.nt; ti++) {
        const GatherTable T = a.t[ti];
        const int W = T.words;
        for (int64_t r0 = wave * kRows; r0 < n; r0 += waves * kRows) {
            // one load brings the kRows keys (lane u holds row r0 + u's), each
            // then broadcast from its lane: loaded one by one, every key would
            // wait for the one before
            int64_t kl = -1;
            if (lane < kRows) {
                const int64_t row = r0 + lane;
                if (row < n) {
                    const int64_t k = T.key == TGL_KEY_NODE ? static_cast<int64_t>(a.nbr[row]) : a.eid[row];
                    kl = k >= 0 && k < T.num_rows ? k : -1;
                }
            }
            int64_t key[kRows];
#pragma unroll
            for (int u = 0; u < kRows; u++) {
                const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(kl), u));
                const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(kl >> 32), u));
                key[u] = static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
            }
            for (int w0 = 0; w0 < W; w0 += kWave) {
                const int w = w0 + lane;
                i32x4 v[kRows];
#pragma unroll
                for (int u = 0; u < kRows; u++)
                    v[u] = key[u] >= 0 && w < W ? T.rows[key[u] * W + w] : zero;
#pragma unroll
                for (int u = 0; u < kRows; u++) {
                    const int64_t row = r0 + u;
                    if (row < n && w < W) __builtin_nontemporal_store(v[u], T.out + row * W + w);
                }
            }
        }
    }
}

}  // namespace
}  // namespace tgl

using namespace tgl;

extern "C" {

tgl_status tgl_gather(const int32_t *nbr, const int64_t *eid, int64_t n, const int64_t *count,
                      int64_t per_count, const tgl_table *tables, int32_t num_tables, void *stream) {
    if (n < 0 || per_count < 1 || !tables || num_tables < 1 || num_tables > TGL_MAX_TABLES) return TGL_EINVAL;
    GatherArgs a{};
    a.nbr = nbr;
    a.eid = eid;
    a.n = n;
    a.count = count;
    a.per = per_count;
    a.nt = num_tables;
    for (int i = 0; i < num_tables; i++) {
        const tgl_table &t = tables[i];
        if (t.row_bytes < 16 || t.row_bytes > TGL_MAX_ROW_BYTES || t.row_bytes % 16 != 0) return TGL_EINVAL;
        if (t.num_rows < 0 || t.num_rows > INT64_MAX / t.row_bytes) return TGL_EINVAL;
        if (t.key != TGL_KEY_NODE && t.key != TGL_KEY_EDGE) return TGL_EINVAL;
        if (n > 0 && !t.out) return TGL_EINVAL;
        if (t.num_rows > 0 && !t.rows) return TGL_EINVAL;
        if ((reinterpret_cast<uintptr_t>(t.rows) & 15u) != 0 || (reinterpret_cast<uintptr_t>(t.out) & 15u) != 0)
            return TGL_EINVAL;
        if (n > 0 && t.key == TGL_KEY_NODE && !nbr) return TGL_EINVAL;
        if (n > 0 && t.key == TGL_KEY_EDGE && !eid) return TGL_EINVAL;
        a.t[i].rows = static_cast<const i32x4 *>(t.rows);
        a.t[i].out = static_cast<i32x4 *>(t.out);
        a.t[i].num_rows = t.num_rows;
        a.t[i].words = t.row_bytes / 16;
        a.t[i].key = t.key;
    }
    if (n == 0) return TGL_OK;
    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    constexpr int64_t rows_per_block = static_cast<int64_t>(kBlock / kWave) * kRows;
    int64_t blocks = (n + rows_per_block - 1) / rows_per_block;
    if (blocks > (1 << 16)) blocks = 1 << 16;
    {
        ScopedTimer tm(TGL_TIMER_GATHER, st);
        gather_kernel<<<static_cast<unsigned>(blocks), kBlock, 0, st>>>(a);
    }
    return launch_status();
}

}  // extern "C"
