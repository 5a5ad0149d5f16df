// tgl_mfg.hip -- one hop's sampled slots as a message-flow-graph block in
// compressed sparse column form (Algorithm 1 of TGL ends every layer with
// "generate DGL MFGs"; the sampler breakdown of Section 4 counts that step as
// "Oth.").
//
// The block is a relabelling of the slot arrays: destinations are the hop's
// groups, edges its valid slots, sources the destinations followed by one
// temporal node per edge.  Its one non-local quantity is each group's first
// edge, the exclusive scan of the per-group valid counts, so the export is
// four passes that never leave the device: per-group valid counts (with the
// destination nodes) and their totals per tile of kScanTile groups, the scan
// of the tile totals, each group's first edge (indptr), and a copy of the
// valid slots, one thread per slot.  A group's valid slots are a prefix of its k slots (tgl_sample
// fills a group newest-first or all-or-nothing); slots after a group's first
// PAD are not exported.
#include "tgl_internal.hpp"

namespace tgl {
namespace {

// G = min(count * windows, cap), from the device count
__device__ __forceinline__ int64_t mfg_groups(const int64_t *count, int64_t windows, int64_t cap) {
    int64_t c = *count;
    c = c < 0 ? 0 : c;
    return c > cap / windows ? cap : c * windows;
}

// Pass 1, one tile of kScanTile groups per block, thread t owning groups
// tile + t, tile + t + 256, ... (neighbouring lanes, neighbouring groups):
// each group's valid prefix length and its destination node (hop 1: the
// group's root; later hops: the previous hop's slot it came from), and the
// tile's edge total.
__global__ __launch_bounds__(kBlock) void mfg_count_kernel(const int32_t *__restrict__ nbr, int32_t k,
                                                           const int32_t *__restrict__ roots,
                                                           const float *__restrict__ root_ts, int32_t windows,
                                                           const int32_t *__restrict__ prev_nbr,
                                                           const float *__restrict__ prev_ts,
                                                           const int64_t *__restrict__ parent,
                                                           const int64_t *__restrict__ count, int64_t cap,
                                                           int64_t *__restrict__ sizes, int32_t *__restrict__ cnt,
                                                           int64_t *__restrict__ partials,
                                                           int32_t *__restrict__ src_nid, float *__restrict__ src_ts) {
    __shared__ int64_t lds[kBlock / kWave];
    const int64_t G = mfg_groups(count, windows, cap);
    if (blockIdx.x == 0 && threadIdx.x == 0) sizes[0] = G;
    const int64_t tile0 = static_cast<int64_t>(blockIdx.x) * kScanTile;
    int64_t sum = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; i++) {
        const int64_t g = tile0 + i * kBlock + threadIdx.x;
        if (g >= G) continue;
        // valid prefix length: slots are read eight at a time, all in flight,
        // and the first PAD among them ends the prefix
        const int32_t *sl = nbr + g * k;
        int32_t c = 0;
        for (int32_t j0 = 0; j0 < k; j0 += 8) {
            int32_t v[8];
#pragma unroll
            for (int u = 0; u < 8; u++) v[u] = sl[j0 + u < k ? j0 + u : k - 1];   // clamped: loads issue together
#pragma unroll
            for (int u = 0; u < 8; u++)
                if (j0 + u >= k) v[u] = -1;
            int32_t run = 8;
#pragma unroll
            for (int u = 7; u >= 0; u--)
                if (v[u] < 0) run = u;
            c += run;
            if (run < 8) break;
        }
        cnt[g] = c;
        sum += c;
        if (prev_nbr) {
            const int64_t p = parent[g];
            src_nid[g] = prev_nbr[p];
            src_ts[g] = prev_ts[p];
        } else if (roots) {
            const int64_t r = g / windows;
            src_nid[g] = roots[r];
            src_ts[g] = root_ts[r];
        } else {                                    // no roots given for a positive count: PAD-like
            src_nid[g] = -1;
            src_ts[g] = -1.0f;
        }
    }
    int64_t total;
    block_exclusive_sum<int64_t>(sum, lds, &total);
    if (threadIdx.x == 0) partials[blockIdx.x] = total;
}

// Slots per lane and round of the scatter: their loads are issued together.
constexpr int kScatterUnroll = 4;

// Pass 4, slots i = g * k + j of the G groups, kScatterUnroll per lane and
// round: valid slot j < cnt[g] becomes edge indptr[g] + j and source node
// G + that edge.  The counts and first edges of a lane's slots are loaded
// together, then their fields; a slot past its group's prefix reads slot 0
// (one cached line) and stores nothing, rather than each load waiting behind
// a branch of its own.  I is the index type (32-bit when the slot capacity
// allows it).  Also closes indptr with indptr[G] = E.
template <class I>
__global__ __launch_bounds__(kBlock) void mfg_scatter_kernel(const int32_t *__restrict__ nbr,
                                                             const int64_t *__restrict__ eid,
                                                             const float *__restrict__ ts,
                                                             const float *__restrict__ dt, int32_t k,
                                                             const int64_t *__restrict__ sizes,
                                                             const int32_t *__restrict__ cnt,
                                                             int64_t *__restrict__ indptr,
                                                             int64_t *__restrict__ edge_dst,
                                                             int64_t *__restrict__ edge_eid,
                                                             float *__restrict__ edge_dt, int32_t *__restrict__ src_nid,
                                                             float *__restrict__ src_ts) {
    constexpr int U = kScatterUnroll;
    const int64_t G = sizes[0];
    if (blockIdx.x == 0 && threadIdx.x == 0) indptr[G] = sizes[1];
    const I total = static_cast<I>(G) * static_cast<I>(k);
    const I kk = static_cast<I>(k);
    const I stride = static_cast<I>(gridDim.x) * kBlock * U;
    for (I i0 = static_cast<I>(blockIdx.x) * kBlock * U + threadIdx.x; i0 < total; i0 += stride) {
        I g[U];
        int32_t j[U], c[U];
        int64_t first[U];
#pragma unroll
        for (int u = 0; u < U; u++) {
            const I i = i0 + static_cast<I>(u) * kBlock;
            const I ic = i < total ? i : total - 1;
            g[u] = ic / kk;
            j[u] = static_cast<int32_t>(ic - g[u] * kk);
            c[u] = cnt[g[u]];
            first[u] = indptr[g[u]];
        }
        I at[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; u++) {
            const I i = i0 + static_cast<I>(u) * kBlock;
            ok[u] = i < total && j[u] < c[u];
            at[u] = ok[u] ? i : 0;
        }
        int64_t ve[U];
        float vd[U], vt[U];
        int32_t vn[U];
#pragma unroll
        for (int u = 0; u < U; u++) {
            ve[u] = eid[at[u]];
            vd[u] = dt[at[u]];
            vn[u] = nbr[at[u]];
            vt[u] = ts[at[u]];
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            if (!ok[u]) continue;
            const int64_t e = first[u] + static_cast<int64_t>(j[u]);
            if (edge_dst) edge_dst[e] = static_cast<int64_t>(g[u]);
            edge_eid[e] = ve[u];
            edge_dt[e] = vd[u];
            src_nid[G + e] = vn[u];
            src_ts[G + e] = vt[u];
        }
    }
}

unsigned grid_of(int64_t n) {
    int64_t b = (n + kBlock - 1) / kBlock;
    if (b < 1) b = 1;
    if (b > (1 << 16)) b = 1 << 16;
    return static_cast<unsigned>(b);
}

struct MfgWs {
    int32_t *cnt = nullptr;
    int64_t *partials = nullptr;
    size_t bytes = 0;
};

MfgWs carve_mfg_ws(void *base, int64_t groups_cap) {
    MfgWs w;
    Carver cv(base);
    w.cnt = cv.take<int32_t>(static_cast<size_t>(groups_cap > 0 ? groups_cap : 1));
    w.partials = cv.take<int64_t>(static_cast<size_t>(scan_tiles(groups_cap) + 1));
    w.bytes = cv.size();
    return w;
}

}  // namespace
}  // namespace tgl

using namespace tgl;

extern "C" {

size_t tgl_mfg_workspace(int64_t groups_cap) {
    if (groups_cap < 0) return 0;
    return carve_mfg_ws(nullptr, groups_cap).bytes;
}

tgl_status tgl_mfg_export(const tgl_hop_out *hop, const tgl_hop_out *prev, const int32_t *roots,
                          const float *root_ts, const int64_t *count, int32_t windows, int32_t k,
                          int64_t groups_cap, const tgl_mfg *out, void *workspace, size_t workspace_bytes,
                          void *stream) {
    if (!hop || !out || !count) return TGL_EINVAL;
    if (windows < 1 || windows > TGL_MAX_SNAPSHOTS || k < 1 || k > TGL_MAX_FANOUT) return TGL_EINVAL;
    if (groups_cap < 0 || groups_cap > (int64_t(1) << 62) / (k + 1)) return TGL_EINVAL;
    if (!out->indptr || !out->sizes) return TGL_EINVAL;
    if (groups_cap > 0) {
        if (!hop->nbr || !hop->eid || !hop->ts || !hop->dt) return TGL_EINVAL;
        if (!out->edge_eid || !out->edge_dt || !out->src_nid || !out->src_ts) return TGL_EINVAL;
        // roots are read only for groups below count * windows, a device value:
        // they may be NULL when the call had no roots
        if (prev && (!prev->nbr || !prev->ts || !hop->parent)) return TGL_EINVAL;
        if (!prev && (!roots) != (!root_ts)) return TGL_EINVAL;
    }
    if (prev && windows != 1) return TGL_EINVAL;
    const MfgWs need = carve_mfg_ws(nullptr, groups_cap);
    if (!workspace || workspace_bytes < need.bytes) return TGL_ENOSPACE;
    const MfgWs ws = carve_mfg_ws(workspace, groups_cap);

    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    ScopedTimer tm(TGL_TIMER_MFG, st);
    const int64_t tiles = scan_tiles(groups_cap) > 0 ? scan_tiles(groups_cap) : 1;
    mfg_count_kernel<<<static_cast<unsigned>(tiles), kBlock, 0, st>>>(
        hop->nbr, k, roots, root_ts, windows, prev ? prev->nbr : nullptr, prev ? prev->ts : nullptr,
        prev ? hop->parent : nullptr, count, groups_cap, out->sizes, ws.cnt, ws.partials, out->src_nid, out->src_ts);
    launch_scan_partials(ws.partials, tiles, out->sizes + 1, st);
    scan_apply_kernel<int32_t, int64_t><<<static_cast<unsigned>(tiles), kBlock, 0, st>>>(
        ws.cnt, out->indptr, groups_cap, out->sizes, ws.partials);
    const int64_t slots = groups_cap * k;
    if (slots < (int64_t(1) << 32) - kBlock * 65536ll * kScatterUnroll)   // no 32-bit wrap past the last round
        mfg_scatter_kernel<uint32_t><<<grid_of((slots + kScatterUnroll - 1) / kScatterUnroll), kBlock, 0, st>>>(
            hop->nbr, hop->eid, hop->ts, hop->dt, k, out->sizes, ws.cnt, out->indptr, out->edge_dst, out->edge_eid,
            out->edge_dt, out->src_nid, out->src_ts);
    else
        mfg_scatter_kernel<uint64_t><<<grid_of((slots + kScatterUnroll - 1) / kScatterUnroll), kBlock, 0, st>>>(
            hop->nbr, hop->eid, hop->ts, hop->dt, k, out->sizes, ws.cnt, out->indptr, out->edge_dst, out->edge_eid,
            out->edge_dt, out->src_nid, out->src_ts);
    return launch_status();
}

}  // extern "C"
