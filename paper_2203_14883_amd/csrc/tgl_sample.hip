// tgl_sample.hip -- multi-hop temporal neighbour sampler over a T-CSR
// (Algorithm 1 and Section 3.1 "Sampling" / "Parallel Sampling" of TGL).
//
// The paper's CPU sampler parallelises over roots with threads and keeps
// per-node pointer arrays that advance with chronological roots; binary search
// is its fallback for layers >= 2.  On the GPU every root is served by a group
// of G lanes of one wavefront, with no shared mutable state:
//
//   1. window location: a G-ary search over the root's time-sorted run (G
//      probes per round, combined with one ballot), so a run of d entries takes
//      about log_{G+1}(d) dependent loads instead of log_2(d);
//   2. selection: lane j of the group takes slot j (most recent: the j-th
//      newest candidate; uniform: a counter-hash draw keyed by the root's path);
//   3. gather + emit: one aligned 16-byte load of the T-CSR entry per slot,
//      and structure-of-arrays stores of (nbr, eid, ts, dt);
//   4. compaction: valid slots form a prefix of every (root, window) group, so
//      a device-wide scan over per-group counts gives each next-hop root its
//      index; the emit step writes the next hop's roots and parent indices.
//
// Nothing is synchronised with the host: per-hop root counts stay on the
// device and the next hop's kernels read them.
#include "tgl_internal.hpp"

namespace tgl {
namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr int kMaxGrid = 1 << 16;     // cap on blocks of the grid-stride hop kernels

__host__ __device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

struct HopArgs {
    // graph
    const int64_t *indptr;
    const int4 *ent;          // tgl_entry viewed as 16-byte vectors
    int64_t num_nodes;
    int64_t num_entries;
    // roots of this hop
    const int32_t *rx;
    const float *rt;
    const int32_t *rs;        // inherited window (hops >= 2), null on hop 1
    const uint64_t *rpath;    // path of each root (hops >= 2), null on hop 1
    uint64_t root_base;
    int64_t count_static;
    const int64_t *count_dyn; // number of roots, read on the device (hops >= 2)
    // parameters
    int32_t hop;              // 1-based
    int32_t k;
    int32_t windows;          // windows per root: S on hop 1, 1 afterwards
    float delta;
    int32_t delta_inf;
    uint64_t seedmix;         // mix64(seed ^ golden)
    // outputs
    int32_t *o_nbr;
    int64_t *o_eid;
    float *o_ts;
    float *o_dt;
    int32_t *o_cnt;           // valid slots per (root, window) group, or null
    int64_t *count0_out;      // hop 1 stores its root count here
};

__device__ __forceinline__ float entry_ts(const int4 *ent, int64_t p) {
    return __int_as_float(reinterpret_cast<const int *>(ent + p)[1]);
}

// Number of entries p in [lo, hi) of a time-sorted run with (double)ts[p] < v,
// found by the G lanes of one group together.  Each round probes G evenly
// spaced positions; the probes below v form a prefix, whose length narrows the
// range to one gap.  A NaN bound compares false everywhere and gives lo.
template <int G>
__device__ __forceinline__ int64_t count_below(const int4 *__restrict__ ent, int64_t lo, int64_t hi,
                                               double v, int gl) {
    while (hi - lo > G) {
        const int64_t len = hi - lo;
        const int64_t pos = lo + (static_cast<int64_t>(gl + 1) * len) / (G + 1);
        const bool below = static_cast<double>(entry_ts(ent, pos)) < v;
        const int c = __popcll(group_ballot<G>(below));
        const int64_t nlo = c > 0 ? lo + (static_cast<int64_t>(c) * len) / (G + 1) + 1 : lo;
        const int64_t nhi = c < G ? lo + (static_cast<int64_t>(c + 1) * len) / (G + 1) : hi;
        lo = nlo;
        hi = nhi;
    }
    const int64_t pos = lo + gl;
    const bool below = pos < hi && static_cast<double>(entry_ts(ent, pos)) < v;
    return lo + __popcll(group_ballot<G>(below));
}

__device__ __forceinline__ double bound_value(float t, int32_t i, float delta) {
    // upper edge of window i (= lower edge of window i - 1): t - i * delta
    return i == 0 ? static_cast<double>(t)
                  : static_cast<double>(t) - static_cast<double>(i) * static_cast<double>(delta);
}

template <bool LAST>
__device__ __forceinline__ void emit_slot(const HopArgs &p, int64_t o, int64_t pick, float t) {
    int32_t nbr = -1;
    int64_t eid = -1;
    float ts = -1.0f, dt = -1.0f;
    if (pick >= 0) {
        const int4 v = p.ent[pick];
        nbr = v.x;
        ts = __int_as_float(v.y);
        eid = static_cast<int64_t>(static_cast<uint32_t>(v.z)) |
              (static_cast<int64_t>(v.w) << 32);
        dt = static_cast<float>(static_cast<double>(t) - static_cast<double>(ts));
    }
    if constexpr (LAST) {
        __builtin_nontemporal_store(nbr, p.o_nbr + o);
        __builtin_nontemporal_store(eid, p.o_eid + o);
        __builtin_nontemporal_store(ts, p.o_ts + o);
        __builtin_nontemporal_store(dt, p.o_dt + o);
    } else {
        p.o_nbr[o] = nbr;
        p.o_eid[o] = eid;
        p.o_ts[o] = ts;
        p.o_dt[o] = dt;
    }
}

// One group of G lanes per root; MULTI: hop-1 roots with S > 1 windows (the
// window edges live in LDS), otherwise one window per root in registers.
template <int G, int MODE, bool MULTI, bool LAST>
__global__ __launch_bounds__(kBlock) void hop_kernel(const HopArgs p) {
    constexpr int GPB = kBlock / G;
    const int gl = threadIdx.x & (G - 1);
    const int grp = threadIdx.x / G;
    __shared__ int64_t edges[MULTI ? GPB * (TGL_MAX_SNAPSHOTS + 1) : 1];
    int64_t *my_edges = edges + (MULTI ? grp * (TGL_MAX_SNAPSHOTS + 1) : 0);

    const int64_t count = p.count_dyn ? *p.count_dyn : p.count_static;
    if (p.count0_out && blockIdx.x == 0 && threadIdx.x == 0) *p.count0_out = count;
    const int64_t M = p.num_entries;
    const int W = p.windows;
    const int k = p.k;

    for (int64_t q = static_cast<int64_t>(blockIdx.x) * GPB + grp; q < count;
         q += static_cast<int64_t>(gridDim.x) * GPB) {
        const int32_t x = p.rx[q];
        const float t = p.rt[q];
        const int32_t s0 = p.rs ? p.rs[q] : 0;
        const uint64_t path = p.rpath ? p.rpath[q] : p.root_base + static_cast<uint64_t>(q);

        int64_t a = 0, b = 0;
        if (x >= 0 && x < p.num_nodes) {
            a = p.indptr[x];
            b = p.indptr[x + 1];
            a = a < 0 ? 0 : (a > M ? M : a);
            b = b < a ? a : (b > M ? M : b);
        }

        int64_t lo = a, hi = a;
        if constexpr (MULTI) {
            // edges i = 0..W: window s spans [edge s+1, edge s)
            for (int i = 0; i <= W; i++) {
                const int64_t c = count_below<G>(p.ent, a, b, bound_value(t, i, p.delta), gl);
                if (gl == 0) my_edges[i] = c;
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        } else {
            hi = count_below<G>(p.ent, a, b, bound_value(t, s0, p.delta), gl);
            if (!p.delta_inf) lo = count_below<G>(p.ent, a, b, bound_value(t, s0 + 1, p.delta), gl);
            if (lo > hi) lo = hi;
        }

        const uint64_t hp = MODE == TGL_UNIFORM ? mix64(p.seedmix ^ path) : 0;
        const int64_t obase = q * static_cast<int64_t>(W) * k;
        for (int e = gl; e < W * k; e += G) {
            int s, j;
            int64_t wlo, whi;
            if constexpr (MULTI) {
                s = e / k;
                j = e - s * k;
                whi = my_edges[s];
                wlo = my_edges[s + 1];
                if (wlo > whi) wlo = whi;
            } else {
                s = s0;
                j = e;
                whi = hi;
                wlo = lo;
            }
            const int64_t n = whi - wlo;
            int64_t pick = -1;
            if constexpr (MODE == TGL_MOST_RECENT) {
                if (j < n) pick = whi - 1 - j;
            } else {
                if (n > 0) {
                    const uint64_t key = (static_cast<uint64_t>(p.hop) << 40) |
                                         (static_cast<uint64_t>(s) << 24) | static_cast<uint64_t>(j);
                    pick = wlo + static_cast<int64_t>(__umul64hi(mix64(hp ^ key), static_cast<uint64_t>(n)));
                }
            }
            emit_slot<LAST>(p, obase + e, pick, t);
        }

        if (p.o_cnt) {
            for (int w = gl; w < W; w += G) {
                int64_t whi = MULTI ? my_edges[w] : hi;
                int64_t wlo = MULTI ? my_edges[w + 1] : lo;
                if (wlo > whi) wlo = whi;
                const int64_t n = whi - wlo;
                const int32_t c = MODE == TGL_MOST_RECENT ? static_cast<int32_t>(n < k ? n : k)
                                                          : (n > 0 ? k : 0);
                p.o_cnt[q * W + w] = c;
            }
        }
        if constexpr (MULTI) {
            // the next root of this group rewrites my_edges
            __builtin_amdgcn_wave_barrier();
        }
    }
}

struct EmitArgs {
    const int32_t *cnt;       // valid slots per group of hop h
    const int64_t *partials;  // exclusive tile offsets
    int64_t n_static;
    const int64_t *n_dyn;     // number of groups (hops >= 2: roots of hop h)
    int32_t k;                // fanout of hop h
    int32_t windows;          // S on hop 1, else 1
    int32_t hop;              // h
    uint64_t root_base;
    // hop-h slots and roots
    const int32_t *h_nbr;
    const float *h_ts;
    const int32_t *h_rs;      // hop >= 2: window of each hop-h root
    const uint64_t *h_rpath;  // hop >= 2: path of each hop-h root
    // next-hop roots
    int32_t *nx;
    float *nt;
    int32_t *ns;
    uint64_t *npath;
    int64_t *parent;
};

// Exclusive offsets of the per-group counts, then one next-hop root per valid
// slot: group g holds slots g*k .. g*k + cnt[g] - 1 (valid slots are a prefix).
__global__ __launch_bounds__(kBlock) void compact_emit_kernel(const EmitArgs p) {
    __shared__ int64_t lds[kBlock / kWave];
    const int64_t n = p.n_dyn ? *p.n_dyn : p.n_static;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile +
                         static_cast<int64_t>(threadIdx.x) * kScanItems;
    int32_t c[kScanItems];
    int64_t sum = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; i++) {
        const int64_t g = base + i;
        c[i] = g < n ? p.cnt[g] : 0;
        sum += c[i];
    }
    int64_t total;
    int64_t q = block_exclusive_sum<int64_t>(sum, lds, &total) + p.partials[blockIdx.x];
    const uint64_t S = static_cast<uint64_t>(p.windows);
    const uint64_t k = static_cast<uint64_t>(p.k);
#pragma unroll
    for (int i = 0; i < kScanItems; i++) {
        const int64_t g = base + i;
        if (g >= n) break;
        int32_t s;
        uint64_t child0;   // path of the child of slot j is child0 + j
        if (p.hop == 1) {
            const uint64_t r = static_cast<uint64_t>(g) / S;
            s = static_cast<int32_t>(static_cast<uint64_t>(g) - r * S);
            child0 = (p.root_base + r) * S * k + static_cast<uint64_t>(s) * k;
        } else {
            s = p.h_rs[g];
            child0 = p.h_rpath[g] * k;
        }
        for (int j = 0; j < c[i]; j++) {
            const int64_t slot = g * p.k + j;
            p.nx[q] = p.h_nbr[slot];
            p.nt[q] = p.h_ts[slot];
            p.ns[q] = s;
            p.npath[q] = child0 + static_cast<uint64_t>(j);
            p.parent[q] = slot;
            q++;
        }
    }
}

template <int G, int MODE, bool MULTI, bool LAST>
void launch_hop_g(const HopArgs &a, int64_t groups_cap, hipStream_t st) {
    constexpr int GPB = kBlock / G;
    int64_t blocks = (groups_cap + GPB - 1) / GPB;
    if (blocks < 1) blocks = 1;
    if (blocks > kMaxGrid) blocks = kMaxGrid;
    hop_kernel<G, MODE, MULTI, LAST><<<static_cast<unsigned>(blocks), kBlock, 0, st>>>(a);
}

template <int MODE, bool MULTI, bool LAST>
void launch_hop_m(int G, const HopArgs &a, int64_t cap, hipStream_t st) {
    switch (G) {
        case 8: launch_hop_g<8, MODE, MULTI, LAST>(a, cap, st); break;
        case 16: launch_hop_g<16, MODE, MULTI, LAST>(a, cap, st); break;
        case 32: launch_hop_g<32, MODE, MULTI, LAST>(a, cap, st); break;
        default: launch_hop_g<64, MODE, MULTI, LAST>(a, cap, st); break;
    }
}

void launch_hop(int G, int mode, bool multi, bool last, const HopArgs &a, int64_t cap, hipStream_t st) {
    if (mode == TGL_MOST_RECENT) {
        if (multi) {
            last ? launch_hop_m<TGL_MOST_RECENT, true, true>(G, a, cap, st)
                 : launch_hop_m<TGL_MOST_RECENT, true, false>(G, a, cap, st);
        } else {
            last ? launch_hop_m<TGL_MOST_RECENT, false, true>(G, a, cap, st)
                 : launch_hop_m<TGL_MOST_RECENT, false, false>(G, a, cap, st);
        }
    } else {
        if (multi) {
            last ? launch_hop_m<TGL_UNIFORM, true, true>(G, a, cap, st)
                 : launch_hop_m<TGL_UNIFORM, true, false>(G, a, cap, st);
        } else {
            last ? launch_hop_m<TGL_UNIFORM, false, true>(G, a, cap, st)
                 : launch_hop_m<TGL_UNIFORM, false, false>(G, a, cap, st);
        }
    }
}

// lanes per root: the slot count rounded up to a power of two, in [8, 64]
int pick_group(int64_t slots_per_root) {
    int g = 8;
    while (g < 64 && g < slots_per_root) g <<= 1;
    return g;
}

constexpr int64_t kCapLimit = int64_t(1) << 62;

// capacities: cap[0] = R, cap[h] = slots of hop h
bool capacities(int64_t R, int32_t hops, const int32_t *fanouts, int32_t S, int64_t *cap) {
    cap[0] = R;
    int64_t c = R;
    if (c > kCapLimit / S) return false;
    c *= S;
    for (int h = 1; h <= hops; h++) {
        if (c > kCapLimit / fanouts[h - 1]) return false;
        c *= fanouts[h - 1];
        cap[h] = c;
    }
    return true;
}

bool sample_args_ok(int64_t R, int32_t hops, const int32_t *fanouts, int32_t S) {
    if (R < 0 || hops < 1 || hops > TGL_MAX_HOPS || !fanouts) return false;
    if (S < 1 || S > TGL_MAX_SNAPSHOTS) return false;
    for (int h = 0; h < hops; h++)
        if (fanouts[h] < 1 || fanouts[h] > TGL_MAX_FANOUT) return false;
    return true;
}

struct SampleWs {
    int32_t *cnt = nullptr;
    int64_t *partials = nullptr;
    int32_t *nx[2] = {nullptr, nullptr};
    float *nt[2] = {nullptr, nullptr};
    int32_t *ns[2] = {nullptr, nullptr};
    uint64_t *npath[2] = {nullptr, nullptr};
    size_t bytes = 0;
};

// Workspace: per-group counts and tile partials (largest hop h < L), and one
// (two when L >= 3) buffers of next-hop roots sized for the largest hop >= 2.
SampleWs carve_sample_ws(void *base, int32_t hops, const int64_t *cap, int32_t S) {
    SampleWs w;
    Carver cv(base);
    if (hops >= 2) {
        int64_t max_groups = cap[0] * S;      // hop-1 groups
        int64_t max_roots = 0;                 // roots of hops 2..L
        for (int h = 2; h <= hops; h++) {
            max_roots = cap[h - 1] > max_roots ? cap[h - 1] : max_roots;
            if (h < hops) max_groups = cap[h - 1] > max_groups ? cap[h - 1] : max_groups;
        }
        w.cnt = cv.take<int32_t>(static_cast<size_t>(max_groups));
        w.partials = cv.take<int64_t>(static_cast<size_t>(scan_tiles(max_groups) + 1));
        const int nbuf = hops >= 3 ? 2 : 1;
        for (int i = 0; i < nbuf; i++) {
            w.nx[i] = cv.take<int32_t>(static_cast<size_t>(max_roots));
            w.nt[i] = cv.take<float>(static_cast<size_t>(max_roots));
            w.ns[i] = cv.take<int32_t>(static_cast<size_t>(max_roots));
            w.npath[i] = cv.take<uint64_t>(static_cast<size_t>(max_roots));
        }
    }
    w.bytes = cv.size();
    if (w.bytes == 0) w.bytes = 256;
    return w;
}

}  // namespace
}  // namespace tgl

using namespace tgl;

extern "C" {

int64_t tgl_sample_capacity(int64_t num_roots, int32_t hops, const int32_t *fanouts,
                            int32_t num_snapshots, int32_t hop) {
    if (!sample_args_ok(num_roots, hops, fanouts, num_snapshots) || hop < 0 || hop > hops) return -1;
    int64_t cap[TGL_MAX_HOPS + 1];
    if (!capacities(num_roots, hops, fanouts, num_snapshots, cap)) return -1;
    return cap[hop];
}

size_t tgl_sample_workspace(int64_t num_roots, int32_t hops, const int32_t *fanouts,
                            int32_t num_snapshots) {
    if (!sample_args_ok(num_roots, hops, fanouts, num_snapshots)) return 0;
    int64_t cap[TGL_MAX_HOPS + 1];
    if (!capacities(num_roots, hops, fanouts, num_snapshots, cap)) return 0;
    return carve_sample_ws(nullptr, hops, cap, num_snapshots).bytes;
}

tgl_status tgl_sample(const tgl_tcsr *g, const int32_t *roots, const float *root_ts,
                      int64_t num_roots, int32_t hops, const int32_t *fanouts, int32_t mode,
                      int32_t num_snapshots, float snapshot_len, uint64_t seed,
                      uint64_t root_base, const tgl_hop_out *outs, int64_t *counts,
                      void *workspace, size_t workspace_bytes, void *stream) {
    // ---- host-side argument checks (nothing is enqueued on failure) ----
    if (!g || !outs || !counts) return TGL_EINVAL;
    if (!sample_args_ok(num_roots, hops, fanouts, num_snapshots)) return TGL_EINVAL;
    if (mode != TGL_MOST_RECENT && mode != TGL_UNIFORM) return TGL_EINVAL;
    if (snapshot_len != snapshot_len || !(snapshot_len > 0.0f)) return TGL_EINVAL;
    const bool dinf = __builtin_isinf(snapshot_len);
    if (dinf && num_snapshots != 1) return TGL_EINVAL;
    if (g->num_nodes < 1 || g->num_nodes > INT32_MAX || g->num_entries < 0) return TGL_EINVAL;
    if (!g->indptr || (g->num_entries > 0 && !g->entries)) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(g->entries) & 15u) != 0) return TGL_EINVAL;
    if (num_roots > 0 && (!roots || !root_ts)) return TGL_EINVAL;
    int64_t cap[TGL_MAX_HOPS + 1];
    if (!capacities(num_roots, hops, fanouts, num_snapshots, cap)) return TGL_EINVAL;
    for (int h = 0; h < hops; h++) {
        const tgl_hop_out &o = outs[h];
        if (cap[h + 1] > 0 && (!o.nbr || !o.eid || !o.ts || !o.dt)) return TGL_EINVAL;
        if (h > 0 && cap[h] > 0 && !o.parent) return TGL_EINVAL;
    }
    const SampleWs need = carve_sample_ws(nullptr, hops, cap, num_snapshots);
    if (hops >= 2 && (!workspace || workspace_bytes < need.bytes)) return TGL_ENOSPACE;
    const SampleWs ws = carve_sample_ws(workspace, hops, cap, num_snapshots);

    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();   // clear a stale error so launch checks are ours

    HopArgs a{};
    a.indptr = g->indptr;
    a.ent = reinterpret_cast<const int4 *>(g->entries);
    a.num_nodes = g->num_nodes;
    a.num_entries = g->num_entries;
    a.root_base = root_base;
    a.delta = snapshot_len;
    a.delta_inf = dinf ? 1 : 0;
    a.seedmix = mix64(seed ^ kGolden);

    const int32_t S = num_snapshots;
    for (int h = 1; h <= hops; h++) {
        const bool last = h == hops;
        const int32_t k = fanouts[h - 1];
        const tgl_hop_out &o = outs[h - 1];
        const int buf = (h - 2) & 1;          // next-root buffer holding hop-h roots (h >= 2)
        a.hop = h;
        a.k = k;
        a.windows = h == 1 ? S : 1;
        a.o_nbr = o.nbr;
        a.o_eid = o.eid;
        a.o_ts = o.ts;
        a.o_dt = o.dt;
        a.o_cnt = last ? nullptr : ws.cnt;
        if (h == 1) {
            a.rx = roots;
            a.rt = root_ts;
            a.rs = nullptr;
            a.rpath = nullptr;
            a.count_static = num_roots;
            a.count_dyn = nullptr;
            a.count0_out = counts;
        } else {
            a.rx = ws.nx[buf];
            a.rt = ws.nt[buf];
            a.rs = ws.ns[buf];
            a.rpath = ws.npath[buf];
            a.count_static = 0;
            a.count_dyn = counts + (h - 1);
            a.count0_out = nullptr;
        }
        const bool multi = h == 1 && S > 1;
        const int G = pick_group(static_cast<int64_t>(a.windows) * k);
        {
            ScopedTimer tm(h == 1 ? TGL_TIMER_HOP1 : TGL_TIMER_HOPN, st);
            launch_hop(G, mode, multi, last, a, cap[h - 1], st);
        }
        if (launch_status() != TGL_OK) return TGL_EDEVICE;
        if (last) break;

        // ---- compaction: hop-h valid slots -> hop-(h+1) roots ----
        const int64_t groups_cap = h == 1 ? cap[0] * S : cap[h - 1];
        const int64_t *groups_dyn = h == 1 ? nullptr : counts + (h - 1);
        const int64_t tiles = scan_tiles(groups_cap) > 0 ? scan_tiles(groups_cap) : 1;
        const int nb = (h - 1) & 1;           // buffer receiving hop-(h+1) roots
        ScopedTimer tm(TGL_TIMER_COMPACT, st);
        scan_reduce_kernel<int32_t><<<static_cast<unsigned>(tiles), kBlock, 0, st>>>(
            ws.cnt, groups_cap, groups_dyn, ws.partials);
        launch_scan_partials(ws.partials, tiles, counts + h, st);
        EmitArgs e{};
        e.cnt = ws.cnt;
        e.partials = ws.partials;
        e.n_static = groups_cap;
        e.n_dyn = groups_dyn;
        e.k = k;
        e.windows = a.windows;
        e.hop = h;
        e.root_base = root_base;
        e.h_nbr = o.nbr;
        e.h_ts = o.ts;
        e.h_rs = h == 1 ? nullptr : ws.ns[buf];
        e.h_rpath = h == 1 ? nullptr : ws.npath[buf];
        e.nx = ws.nx[nb];
        e.nt = ws.nt[nb];
        e.ns = ws.ns[nb];
        e.npath = ws.npath[nb];
        e.parent = outs[h].parent;
        compact_emit_kernel<<<static_cast<unsigned>(tiles), kBlock, 0, st>>>(e);
        if (launch_status() != TGL_OK) return TGL_EDEVICE;
    }
    return TGL_OK;
}

}  // extern "C"
