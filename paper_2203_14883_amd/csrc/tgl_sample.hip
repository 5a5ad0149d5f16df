// tgl_sample.hip -- multi-hop temporal neighbour sampler over a T-CSR
// (Algorithm 1 and Section 3.1 "Sampling" / "Parallel Sampling" of TGL).
//
// The paper's CPU sampler parallelises over roots with threads and keeps
// per-node pointer arrays that advance with chronological roots; binary search
// is its fallback for layers >= 2.  On the GPU every root is served by a group
// of G lanes of one wavefront, with no shared mutable state:
//
//   1. window location: the root's run [start, end) and its first and last
//      timestamps come from the node's 16-byte summary; a window edge those
//      decide is not searched.  The search reads only the T-CSR's separate
//      timestamp array.  A short run is loaded whole, 16-byte loads spread over
//      the group's lanes, and every edge is a few ballots over it; a longer
//      run is narrowed G-ary (G probes per round, one ballot), first on the
//      search index (every 32nd timestamp, cache-resident) when the graph has
//      one, so that only the last load of a search reads the run itself.  All
//      edges of one root are searched together: their probes of a round are in
//      flight at once;
//   2. selection: lane j of the group takes slot j (most recent: the j-th
//      newest candidate; uniform: a counter-hash draw keyed by the root's path);
//   3. gather + emit: one aligned 16-byte load of the chosen T-CSR record per
//      slot; slots are written as structure-of-arrays (nbr, eid, ts, dt);
//   4. next hop: valid slots are a prefix of every (root, window) group, so an
//      exclusive scan of the per-group counts gives every next-hop root its
//      index.  The next hop's kernel walks the previous hop's slots directly
//      ("virtual roots"): each wavefront loads 64 of them, compacts the valid
//      ones through LDS, and serves them G lanes per root.  No list of next-hop
//      roots is materialised.
//
// Nothing is synchronised with the host: per-hop root counts stay on the
// device and the next hop's kernels read them.
#include <mutex>

#include "tgl_cells.hpp"
#include "tgl_internal.hpp"

namespace tgl {
namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
constexpr int kMaxGrid = 1 << 16;      // cap on blocks of the grid-stride hop kernels
constexpr int kMultiEdges = 9;       // window edges per root held in LDS by hop_multi_kernel (S <= 8)
constexpr int kWavesPerBlock = kBlock / kWave;

__host__ __device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

struct HopArgs {
    // graph
    const int64_t *indptr;
    const int4 *ent;            // tgl_entry viewed as 16-byte vectors
    const float *tsa;           // timestamps of the entries (search array)
    const float *tsx;           // search index: every TGL_INDEX_STRIDE-th timestamp, or null
    uint32_t nx;                // its length
    const int4 *nodes;          // tgl_node per node (8 x 16 bytes): run start, end, first ts,
                                // last ts, then the run's first timestamps
    const uint2 *hist;          // tgl_span per entry: the neighbour's entries older than it
    const uint2 *dir;           // tgl_cell per search-index slot: the runs' time directories, or null
    int64_t num_nodes;
    int64_t num_entries;
    // hop 1: dense roots
    const int32_t *rx;
    const float *rt;
    int64_t num_roots;
    // hops >= 2: the previous hop's slots are the candidate roots
    const int32_t *p_nbr;
    const float *p_ts;
    const int32_t *p_local;     // previous hop's groups: exclusive offset within the scan tile ...
    const int64_t *p_tile;      // ... plus the exclusive offset of the tile (kScanTile groups)
    const int32_t *p_s;         // window of each previous-hop group (null: hop 1 groups)
    const float *p_t0;          // hop-1 ancestor time of each previous-hop group (anchor A, hops >= 3)
    const uint64_t *p_path;     // path of each previous-hop group (null: hop 1 groups)
    int32_t p_k;                // fanout of the previous hop
    int64_t p_groups_static;    // previous hop's groups (hop 1 groups: R*S) ...
    const int64_t *p_groups_dyn; // ... or read on the device (roots of hop >= 2)
    const uint8_t *p_first;     // TGL_NBR_FIRST hint of each previous-hop slot, or null
    const uint2 *p_win;         // window of each previous-hop slot's root (hist of its entry)
    // parameters
    uint64_t root_base;
    int32_t S;                  // snapshots
    int32_t hop;                // 1-based
    int32_t k;
    int32_t windows;            // windows per root: S on hop 1, 1 afterwards
    float delta;
    int32_t delta_inf;
    int32_t anchor;             // TGL_ANCHOR_OWN / TGL_ANCHOR_ROOT (windows of hops >= 2)
    uint32_t *ptr;              // hop 1: saved window edges, (S + 1) x num_nodes, or null
    uint64_t seedmix;           // mix64(seed ^ golden)
    // outputs
    int32_t *o_nbr;
    int64_t *o_eid;
    float *o_ts;
    float *o_dt;
    int64_t *o_parent;          // hops >= 2
    int32_t *o_cnt;             // valid slots per (root, window) group, or null (last hop)
    int32_t *o_s;               // window of each root, for a later hop (or null)
    float *o_t0;                // hop-1 ancestor time of each root, for a later hop (anchor A, or null)
    uint64_t *o_path;           // path of each root, for a later hop (or null)
    uint8_t *o_first;           // TGL_NBR_FIRST hint of each slot, for the next hop (or null)
    uint2 *o_win;               // hist of each valid slot's entry, for the next hop (WIN kernels)
    int64_t *count0_out;        // hop 1 stores its root count here
};

// ts[p4 .. p4+3] for p4 a multiple of 4; entries at or past M read as +inf
// (they are never inside a window).
__device__ __forceinline__ float4 load_ts4(const float *__restrict__ tsa, uint32_t p4, uint32_t M) {
    if (static_cast<uint64_t>(p4) + 3 < M) return *reinterpret_cast<const float4 *>(tsa + p4);
    const float inf = __builtin_inff();
    float4 r = make_float4(inf, inf, inf, inf);
    if (p4 < M) r.x = tsa[p4];
    if (static_cast<uint64_t>(p4) + 1 < M) r.y = tsa[p4 + 1];
    if (static_cast<uint64_t>(p4) + 2 < M) r.z = tsa[p4 + 2];
    return r;
}

// A stretch of a time-sorted run held in the registers of one G-lane group:
// lane gl holds the H timestamps p0 .. p0 + H - 1, p0 = (lo & ~3) + H * gl,
// loaded as H / 4 aligned float4.  One load covers any [lo, hi) of at most
// `span` entries.
template <int G>
struct HeldRun {
    static constexpr int NV = G >= 16 ? 1 : 16 / G;     // float4 per lane
    static constexpr uint32_t H = 4 * NV;               // timestamps per lane
    static constexpr uint32_t span = H * G - 3;
    float4 v[NV];
    uint32_t p0;
};

template <int G>
__device__ __forceinline__ HeldRun<G> load_run(const float *__restrict__ tsa, uint32_t lo, uint32_t hi,
                                               uint32_t M, int gl) {
    HeldRun<G> r;
    r.p0 = (lo & ~3u) + HeldRun<G>::H * static_cast<uint32_t>(gl);
    const float inf = __builtin_inff();
#pragma unroll
    for (int m = 0; m < HeldRun<G>::NV; m++) {
        const uint32_t p4 = r.p0 + 4 * m;
        r.v[m] = p4 < hi && lo < hi ? load_ts4(tsa, p4, M) : make_float4(inf, inf, inf, inf);
    }
    return r;
}

// The run [a, b), b - a <= TGL_NODE_INLINE, held from the inline timestamps
// of its node record rec (16-byte words 1..7): position a + i is inline
// timestamp i, so the stretch starts at a and count_in applies unchanged.
template <int G>
__device__ __forceinline__ HeldRun<G> load_inline(const int4 *__restrict__ rec, uint32_t a, int gl) {
    constexpr int kWords = TGL_NODE_INLINE / 4;
    static_assert(HeldRun<G>::H * G >= TGL_NODE_INLINE, "held stretch covers the inline timestamps");
    HeldRun<G> r;
    r.p0 = a + HeldRun<G>::H * static_cast<uint32_t>(gl);
    const float inf = __builtin_inff();
#pragma unroll
    for (int m = 0; m < HeldRun<G>::NV; m++) {
        const int q = HeldRun<G>::NV * gl + m;
        if (q < kWords) {
            const int4 w = rec[1 + q];
            r.v[m] = make_float4(__int_as_float(w.x), __int_as_float(w.y), __int_as_float(w.z), __int_as_float(w.w));
        } else {
            r.v[m] = make_float4(inf, inf, inf, inf);
        }
    }
    return r;
}

// Sum over the G lanes of the calling lane's group.
template <int G>
__device__ __forceinline__ int group_sum(int c) {
#pragma unroll
    for (int off = G / 2; off >= 1; off >>= 1) c += __shfl_xor(c, off, kWave);
    return c;
}

// lo + #{p in [lo, hi): ts[p] < v} for [lo, hi) inside the held stretch.
template <int G>
__device__ __forceinline__ uint32_t count_in(const HeldRun<G> &r, uint32_t lo, uint32_t hi, float v) {
    int c = 0;
#pragma unroll
    for (int m = 0; m < HeldRun<G>::NV; m++) {
        const uint32_t p = r.p0 + 4 * m;
        c += (p >= lo && p < hi && r.v[m].x < v);
        c += (p + 1 >= lo && p + 1 < hi && r.v[m].y < v);
        c += (p + 2 >= lo && p + 2 < hi && r.v[m].z < v);
        c += (p + 3 >= lo && p + 3 < hi && r.v[m].w < v);
    }
    return lo + static_cast<uint32_t>(group_sum<G>(c));
}

// For each i: lo[i] += #{p in [lo[i], hi[i]): arr[p] < v[i]}, over a sorted
// stretch of arr (n_arr elements), found by the G lanes of one group together.
// While a range is longer than one held stretch, each round probes G evenly
// spaced positions of it; the probes below v[i] form a prefix, whose length
// narrows the range to one gap; the last range is loaded whole and counted.
// The NE searches advance together, so the probes of one round, and the final
// loads, of all of them are in flight at the same time: the chain of dependent
// loads is that of one search.
template <int G, int NE>
__device__ __forceinline__ void search_n(const float *__restrict__ arr, uint32_t n_arr, uint32_t (&lo)[NE],
                                         uint32_t (&hi)[NE], const float (&v)[NE], int gl) {
    for (;;) {
        bool any = false;
#pragma unroll
        for (int i = 0; i < NE; i++) any |= hi[i] - lo[i] > HeldRun<G>::span;
        if (!any) break;                            // group-uniform
        // probes at lo + j * step, j = 1..G, step = len / (G + 1) >= 1: all
        // inside (lo, hi), strictly increasing
        float probe[NE];
#pragma unroll
        for (int i = 0; i < NE; i++) {
            probe[i] = 0.0f;
            const uint32_t len = hi[i] - lo[i];
            if (len > HeldRun<G>::span)
                probe[i] = arr[lo[i] + static_cast<uint32_t>(gl + 1) * (len / (G + 1))];
        }
#pragma unroll
        for (int i = 0; i < NE; i++) {
            const uint32_t len = hi[i] - lo[i];
            if (len > HeldRun<G>::span) {           // group-uniform
                const uint32_t step = len / (G + 1);
                const uint32_t c = static_cast<uint32_t>(__popcll(group_ballot<G>(probe[i] < v[i])));
                // probes 1..c are below v[i], probe c+1 (if any) is not
                const uint32_t nlo = c > 0 ? lo[i] + c * step + 1 : lo[i];
                if (c < G) hi[i] = lo[i] + (c + 1) * step;
                lo[i] = nlo;
            }
        }
    }
    bool open = false;
#pragma unroll
    for (int i = 0; i < NE; i++) open |= hi[i] > lo[i];
    if (!open) return;                              // group-uniform: every answer is known
    HeldRun<G> r[NE];
#pragma unroll
    for (int i = 0; i < NE; i++) r[i] = load_run<G>(arr, lo[i], hi[i], n_arr, gl);
#pragma unroll
    for (int i = 0; i < NE; i++) lo[i] = count_in<G>(r[i], lo[i], hi[i], v[i]);
}

// A node's run [a, b) and its first and last timestamps: where a threshold
// falls in it is estimated by linear interpolation between them.
struct RunShape {
    uint32_t a, b;
    float first, last;
};

// Estimated position of threshold v in the run (lower bound: the count of
// timestamps below v, plus a), and the spread of that estimate: if the
// run's timestamps were independent draws between first and last, the count
// below v would be binomial, with standard deviation at most sqrt(b - a) / 2.
__device__ __forceinline__ void run_estimate(const RunShape &rs, float v, uint32_t &pos, uint32_t &spread) {
    const float n = static_cast<float>(rs.b - rs.a);
    float f = (v - rs.first) / (rs.last - rs.first);
    if (!(f >= 0.0f)) f = f < 0.0f ? 0.0f : 0.5f;                 // below the run, or NaN
    if (f > 1.0f) f = 1.0f;
    const float o = f * n;                                         // <= n
    pos = rs.a + (o < n ? static_cast<uint32_t>(o) : rs.b - rs.a);
    spread = static_cast<uint32_t>(0.5f * __builtin_sqrtf(n)) + 1u;
}

// Probe g of a guided round: c + (g - G/2) d + d/2, clamped into [lo, hi).
// Non-decreasing in g.
template <int G>
__device__ __forceinline__ uint32_t guided_pos(uint32_t lo, uint32_t hi, uint32_t c, uint32_t d, int g) {
    const int64_t q = static_cast<int64_t>(c) + (static_cast<int64_t>(g) - G / 2) * static_cast<int64_t>(d) +
                      static_cast<int64_t>(d / 2);
    const int64_t last = static_cast<int64_t>(hi) - 1;
    return static_cast<uint32_t>(q < static_cast<int64_t>(lo) ? static_cast<int64_t>(lo) : (q > last ? last : q));
}

// One round of the search of a sorted stretch of arr, guided by estimates:
// for each i whose range [lo[i], hi[i]) is longer than a held stretch, the G
// lanes probe positions d[i] apart around c[i].  The probes below v[i] form
// a prefix (arr is sorted and the positions do not decrease), so the answer
// lies after the last of them and at or before the next: the range shrinks
// to about d[i] when the estimate is off by less than G/2 spacings, and
// never grows.  lo[i] + #{p in [lo[i], hi[i]): arr[p] < v[i]} is unchanged.
template <int G, int NE>
__device__ __forceinline__ void guided_round(const float *__restrict__ arr, uint32_t (&lo)[NE], uint32_t (&hi)[NE],
                                             const float (&v)[NE], const uint32_t (&c)[NE], const uint32_t (&d)[NE],
                                             int gl) {
    float probe[NE];
#pragma unroll
    for (int i = 0; i < NE; i++) {
        probe[i] = 0.0f;
        if (hi[i] - lo[i] > HeldRun<G>::span) probe[i] = arr[guided_pos<G>(lo[i], hi[i], c[i], d[i], gl)];
    }
#pragma unroll
    for (int i = 0; i < NE; i++) {
        if (hi[i] - lo[i] > HeldRun<G>::span) {     // group-uniform
            const int n = __popcll(group_ballot<G>(probe[i] < v[i]));
            const uint32_t nlo = n > 0 ? guided_pos<G>(lo[i], hi[i], c[i], d[i], n - 1) + 1 : lo[i];
            if (n < G) hi[i] = guided_pos<G>(lo[i], hi[i], c[i], d[i], n);
            lo[i] = nlo;
        }
    }
}

// Positions below NE thresholds, each in a range of its own: out[i] = lo0[i]
// + #{p in [lo0[i], hi0[i]): ts[p] < v[i]} for each i with act[i] (lo0[i] otherwise),
// each range a stretch of one sorted run.  Ranges longer than one probe round
// are narrowed on the search index first when there is one.
template <int G, int NE>
__device__ __forceinline__ void count_below_ranges(const float *__restrict__ tsa, uint32_t M,
                                                   const float *__restrict__ tsx, uint32_t nx,
                                                   const uint32_t (&lo0)[NE], const uint32_t (&hi0)[NE],
                                                   const float (&v)[NE], const bool (&act)[NE],
                                                   uint32_t (&out)[NE], int gl) {
    constexpr uint32_t X = TGL_INDEX_STRIDE;
    uint32_t lo[NE], hi[NE];
    bool any_index = false;
#pragma unroll
    for (int i = 0; i < NE; i++) {
        const bool use = act[i] && tsx && hi0[i] - lo0[i] > HeldRun<G>::span * (G + 1);
        const uint32_t ja = lo0[i] / X + (lo0[i] % X != 0);
        const uint32_t jb = hi0[i] / X + (hi0[i] % X != 0);
        lo[i] = use ? ja : lo0[i];
        hi[i] = use ? jb : lo0[i];
        any_index |= use;
    }
    if (any_index) {                                // group-uniform
        search_n<G, NE>(tsx, nx, lo, hi, v, gl);
#pragma unroll
        for (int i = 0; i < NE; i++) {
            const bool use = act[i] && tsx && hi0[i] - lo0[i] > HeldRun<G>::span * (G + 1);
            const uint32_t ja = lo0[i] / X + (lo0[i] % X != 0);
            const uint32_t jb = hi0[i] / X + (hi0[i] % X != 0);
            const uint32_t r = lo[i];
            lo[i] = use ? (r > ja ? (r - 1) * X + 1 : lo0[i]) : lo0[i];   // ts[(r-1) X] < v[i]
            hi[i] = use ? (r < jb ? r * X : hi0[i]) : (act[i] ? hi0[i] : lo0[i]);   // ts[r X] >= v[i]
        }
    } else {
#pragma unroll
        for (int i = 0; i < NE; i++) {
            lo[i] = lo0[i];
            hi[i] = act[i] ? hi0[i] : lo0[i];
        }
    }
    search_n<G, NE>(tsa, M, lo, hi, v, gl);
#pragma unroll
    for (int i = 0; i < NE; i++) out[i] = act[i] ? lo[i] : lo0[i];
}

// Positions below NE thresholds in [lo0, hi0), a range of the run [rs.a,
// rs.b), from the run's time directory (tgl_cell per search-index slot; the
// run owns K >= 1 cells), as count_below_n returns them: threshold i falls in cell
// k = cell(v[i]), whose first position pos and timestamp, and the next
// cell's pos (rs.b after the last cell), are read with one round of loads.
// The run's count below v[i] is pos when v[i] <= ts[pos], else it lies in
// [pos + 1, next pos], a stretch of about TGL_INDEX_STRIDE entries when the
// run's timestamps are spread evenly, which count_below_ranges searches
// (with the index when it is long).  Clamping the stretch into [lo0, hi0)
// gives the count within that range.  Every position read from the
// directory is clamped into the run.
template <int G, int NE>
__device__ __forceinline__ void count_below_dir(const float *__restrict__ tsa, uint32_t M,
                                                const float *__restrict__ tsx, uint32_t nx,
                                                const uint2 *__restrict__ dir, uint32_t lo0, uint32_t hi0,
                                                const RunShape &rs, const float (&v)[NE], const bool (&act)[NE],
                                                uint32_t (&out)[NE], int gl) {
    constexpr uint32_t X = TGL_INDEX_STRIDE;
    const uint32_t ja = rs.a / X + (rs.a % X != 0);
    const uint32_t K = rs.b / X + (rs.b % X != 0) - ja;
    const float sc = dir_scale(rs.first, rs.last, K);
    uint2 c0[NE];
    uint32_t c1[NE];
#pragma unroll
    for (int i = 0; i < NE; i++) {
        c0[i] = make_uint2(rs.a, 0u);
        c1[i] = rs.b;
        if (act[i]) {                               // group-uniform
            const uint32_t kc = dir_cell(v[i], rs.first, rs.last, sc, K);
            c0[i] = dir[ja + kc];
            if (kc + 1 < K) c1[i] = dir[ja + kc + 1].x;
        }
    }
    uint32_t lo[NE], hi[NE];
    bool open[NE];
#pragma unroll
    for (int i = 0; i < NE; i++) {
        const uint32_t pos = c0[i].x < rs.a ? rs.a : (c0[i].x > rs.b ? rs.b : c0[i].x);
        const uint32_t nxt = c1[i] < pos ? pos : (c1[i] > rs.b ? rs.b : c1[i]);
        const bool past = v[i] > __uint_as_float(c0[i].y) && pos < nxt;
        uint32_t l = past ? pos + 1 : pos;
        uint32_t h = past ? nxt : l;
        l = l < lo0 ? lo0 : (l > hi0 ? hi0 : l);
        h = h < l ? l : (h > hi0 ? hi0 : h);
        lo[i] = act[i] ? l : lo0;
        hi[i] = act[i] ? h : lo0;
        open[i] = act[i] && h > l;
    }
    count_below_ranges<G, NE>(tsa, M, tsx, nx, lo, hi, v, open, out, gl);
}

// Positions below NE thresholds in the time-sorted run [lo0, hi0) of the
// timestamp array (M entries): out[i] = lo0 + #{p in [lo0, hi0): ts[p] < v[i]}
// for each i with act[i] (out[i] = lo0 otherwise).  rec, when not null, is the
// record of a node whose whole run (lo0 onwards) is inline in it: the run is
// then read from there.  A run of at most one held stretch is loaded once and
// serves every threshold.  A longer range starts from the time directory dir
// of its run rs when there is one (count_below_dir).  Otherwise a range long
// enough to need more than one probe round is first narrowed on the search
// index tsx (nx samples, tsx[j] = ts[j * TGL_INDEX_STRIDE]) when there is
// one, starting with a round guided by the run shape rs (the run that holds
// the stretch, lo0 its start): with r the samples inside the run below v[i],
// the answer lies after sample r - 1 and at or before sample r, fewer than
// TGL_INDEX_STRIDE timestamps.
template <int G, int NE, bool DIR>
__device__ __forceinline__ void count_below_n(const float *__restrict__ tsa, uint32_t M,
                                              const float *__restrict__ tsx, uint32_t nx,
                                              const uint2 *__restrict__ dir,
                                              const int4 *__restrict__ rec, uint32_t lo0, uint32_t hi0,
                                              const RunShape &rs, const float (&v)[NE], const bool (&act)[NE],
                                              uint32_t (&out)[NE], int gl) {
    constexpr uint32_t X = TGL_INDEX_STRIDE;
    if (rec || hi0 - lo0 <= HeldRun<G>::span) {    // group-uniform: one load serves every bound
        const HeldRun<G> r = rec ? load_inline<G>(rec, lo0, gl) : load_run<G>(tsa, lo0, hi0, M, gl);
#pragma unroll
        for (int i = 0; i < NE; i++) out[i] = act[i] ? count_in<G>(r, lo0, hi0, v[i]) : lo0;
        return;
    }
    if constexpr (DIR) {
        // the range is longer than one held stretch, so its run owns a cell
        count_below_dir<G, NE>(tsa, M, tsx, nx, dir, lo0, hi0, rs, v, act, out, gl);
#pragma unroll
        for (int i = 0; i < NE; i++)
            if (!act[i]) out[i] = lo0;
        return;
    }
    uint32_t lo[NE], hi[NE];
    if (tsx && hi0 - lo0 > HeldRun<G>::span * (G + 1)) {   // group-uniform
        // samples j in [ja, jb) are the positions j * X inside [lo0, hi0)
        const uint32_t ja = lo0 / X + (lo0 % X != 0);
        const uint32_t jb = hi0 / X + (hi0 % X != 0);
        uint32_t gc[NE], gd[NE];
#pragma unroll
        for (int i = 0; i < NE; i++) {
            lo[i] = ja;
            hi[i] = act[i] ? jb : ja;
            uint32_t pos, spread;
            run_estimate(rs, v[i], pos, spread);
            gc[i] = pos / X;
            gd[i] = spread / X > 0 ? spread / X : 1u;
        }
        guided_round<G, NE>(tsx, lo, hi, v, gc, gd, gl);
        search_n<G, NE>(tsx, nx, lo, hi, v, gl);
#pragma unroll
        for (int i = 0; i < NE; i++) {
            const uint32_t r = lo[i];
            lo[i] = r > ja ? (r - 1) * X + 1 : lo0;  // ts[(r-1) X] < v[i]
            hi[i] = r < jb ? r * X : hi0;            // ts[r X] >= v[i]
            if (!act[i]) hi[i] = lo[i];
        }
    } else {
#pragma unroll
        for (int i = 0; i < NE; i++) {
            lo[i] = lo0;
            hi[i] = act[i] ? hi0 : lo0;
        }
    }
    search_n<G, NE>(tsa, M, lo, hi, v, gl);
#pragma unroll
    for (int i = 0; i < NE; i++) out[i] = act[i] ? lo[i] : lo0;
}

// Window edges of a long run [a, b) found from saved positions -- the
// per-node pointers of Section 3.1, kept for hop 1 -- by the G lanes of one
// group: edge i (threshold v[i]) is first looked for in the held stretch that
// starts one entry before its saved position ptr[ei[i] * N + x].  If the whole
// stretch lies at or above v[i] the edge is before it, if the whole stretch
// lies below v[i] the edge is after it: only then is the rest of the run
// searched.  The saved position is raised to the edge found.  Any saved
// position in [a, b] gives the same result; a chronological root stream
// makes the first load the answer.
template <int G, int NE>
__device__ __forceinline__ void from_pointers(const HopArgs &p, int32_t x, uint32_t a, uint32_t b,
                                              const int (&ei)[NE], const float (&v)[NE], const bool (&act)[NE],
                                              uint32_t (&out)[NE], int gl) {
    const uint32_t M = static_cast<uint32_t>(p.num_entries);
    constexpr uint32_t span = HeldRun<G>::span;
    uint32_t lo[NE], hi[NE], saved[NE];
#pragma unroll
    for (int i = 0; i < NE; i++) {
        uint32_t p0 = a;
        saved[i] = 0;
        if (act[i]) {
            saved[i] = p.ptr[static_cast<int64_t>(ei[i]) * p.num_nodes + x];
            p0 = saved[i] < a ? a : (saved[i] > b ? b : saved[i]);
        }
        lo[i] = p0 > a ? p0 - 1 : a;
        hi[i] = act[i] ? (b - lo[i] > span ? lo[i] + span : b) : lo[i];
    }
    HeldRun<G> r[NE];
#pragma unroll
    for (int i = 0; i < NE; i++) r[i] = load_run<G>(p.tsa, lo[i], hi[i], M, gl);
    uint32_t flo[NE], fhi[NE];
    bool fb[NE];
    bool any = false;
#pragma unroll
    for (int i = 0; i < NE; i++) {
        out[i] = count_in<G>(r[i], lo[i], hi[i], v[i]);
        fb[i] = act[i] && ((out[i] == lo[i] && lo[i] > a) || (out[i] == hi[i] && hi[i] < b));
        flo[i] = fb[i] ? (out[i] == lo[i] && lo[i] > a ? a : hi[i]) : a;
        fhi[i] = fb[i] ? (out[i] == lo[i] && lo[i] > a ? lo[i] : b) : a;
        any |= fb[i];
    }
    if (any) {                                      // group-uniform
        uint32_t fo[NE];
        count_below_ranges<G, NE>(p.tsa, M, p.tsx, p.nx, flo, fhi, v, fb, fo, gl);
#pragma unroll
        for (int i = 0; i < NE; i++)
            if (fb[i]) out[i] = fo[i];
    }
    // raise the saved position only when this edge lies beyond it: roots of a
    // hot node mostly find it already there, and skip the atomic
    if (gl == 0) {
#pragma unroll
        for (int i = 0; i < NE; i++)
            if (act[i] && out[i] > saved[i]) atomicMax(p.ptr + static_cast<int64_t>(ei[i]) * p.num_nodes + x, out[i]);
    }
}

// Upper edge of window i (= lower edge of window i - 1), t - i * delta, as a
// float threshold.  Window membership compares a timestamp with the edge
// computed in double; rounding the edge up to the nearest float f >= edge (+inf
// above the float range, NaN for NaN) gives the same answer for every float
// timestamp x: x < edge exactly when x < f, as no float lies in [edge, f).
__device__ __forceinline__ float bound_value(float t, int32_t i, float delta) {
    const double e = i == 0 ? static_cast<double>(t)
                            : static_cast<double>(t) - static_cast<double>(i) * static_cast<double>(delta);
    return __double2float_ru(e);
}

// a + #{p in [a, b): ts[p] < v} when the run's first and last timestamps
// decide it alone (the run is sorted): a if first >= v (or v is NaN), b if
// last < v.  Returns false when the edge falls inside the run.
__device__ __forceinline__ bool edge_from_summary(uint32_t a, uint32_t b, float first, float last, float v,
                                                  uint32_t &c) {
    if (!(first < v)) {
        c = a;
        return true;
    }
    if (last < v) {
        c = b;
        return true;
    }
    return false;
}

struct NodeRun {
    uint32_t a, b;
    float first, last;
};

// Run of node x from its summary record, clamped into [0, M]; an out-of-range
// node has an empty run.
__device__ __forceinline__ NodeRun node_run(const HopArgs &p, int32_t x, bool valid) {
    NodeRun r{0u, 0u, __builtin_inff(), -__builtin_inff()};
    if (valid && x >= 0 && x < p.num_nodes) {
        const int4 nd = p.nodes[static_cast<int64_t>(x) * 8];
        const uint32_t M = static_cast<uint32_t>(p.num_entries);
        uint32_t a = static_cast<uint32_t>(nd.x);
        uint32_t b = static_cast<uint32_t>(nd.y);
        a = a > M ? M : a;
        b = b < a ? a : (b > M ? M : b);
        r.a = a;
        r.b = b;
        r.first = __int_as_float(nd.z);
        r.last = __int_as_float(nd.w);
    }
    return r;
}

// Writes slot o from entry v (valid) or as PAD; the neighbour id loses the
// entry's hint bit, which goes to o_first for the next hop.
template <bool LAST>
__device__ __forceinline__ void emit_slot(const HopArgs &p, int64_t o, bool valid, int4 v, float t) {
    int32_t nbr = -1;
    int64_t eid = -1;
    float ts = -1.0f, dt = -1.0f;
    if constexpr (!LAST) {
        if (p.o_first) p.o_first[o] = valid && v.x < 0 ? 1 : 0;
    }
    if (valid) {
        nbr = static_cast<int32_t>(static_cast<uint32_t>(v.x) & TGL_NBR_MASK);
        ts = __int_as_float(v.y);
        eid = static_cast<int64_t>(static_cast<uint32_t>(v.z)) | (static_cast<int64_t>(v.w) << 32);
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

// Output arrays of one chunk, offset to its first slot: a slot is then
// addressed by a 32-bit offset from a wavefront-uniform base.
struct OutRow {
    int32_t *nbr;
    int64_t *eid;
    float *ts;
    float *dt;
    uint8_t *first;             // TGL_NBR_FIRST hint per slot, or null
    uint2 *win;                 // next hop's window per valid slot, or null
};

// emit_slot for slot e of the chunk whose outputs start at o.
template <bool LAST>
__device__ __forceinline__ void emit_at(const OutRow &o, uint32_t e, bool valid, int4 v, float t) {
    int32_t nbr = -1;
    int64_t eid = -1;
    float ts = -1.0f, dt = -1.0f;
    if constexpr (!LAST) {
        if (o.first) o.first[e] = valid && v.x < 0 ? 1 : 0;
    }
    if (valid) {
        nbr = static_cast<int32_t>(static_cast<uint32_t>(v.x) & TGL_NBR_MASK);
        ts = __int_as_float(v.y);
        eid = static_cast<int64_t>(static_cast<uint32_t>(v.z)) | (static_cast<int64_t>(v.w) << 32);
        dt = static_cast<float>(static_cast<double>(t) - static_cast<double>(ts));
    }
    if constexpr (LAST) {
        __builtin_nontemporal_store(nbr, o.nbr + e);
        __builtin_nontemporal_store(eid, o.eid + e);
        __builtin_nontemporal_store(ts, o.ts + e);
        __builtin_nontemporal_store(dt, o.dt + e);
    } else {
        o.nbr[e] = nbr;
        o.eid[e] = eid;
        o.ts[e] = ts;
        o.dt[e] = dt;
    }
}

// A 64-bit value that is the same in every active lane, moved to scalar
// registers.
__device__ __forceinline__ int64_t uniform64(int64_t v) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(static_cast<uint64_t>(v) >> 32));
    return static_cast<int64_t>((static_cast<uint64_t>(hi) << 32) | lo);
}

// The T-CSR records of U picks (UINT32_MAX: no pick), with all U loads in
// flight together.  A lane without a pick reads entry 0 and its caller
// ignores the record: predicating the loads instead would put each behind a
// branch and a wait of its own.
template <int U>
__device__ __forceinline__ void gather_records(const int4 *__restrict__ ent, uint32_t M, const uint32_t (&pick)[U],
                                               int4 (&rec)[U]) {
    if (M == 0) {                                   // uniform: nothing to read
#pragma unroll
        for (int u = 0; u < U; u++) rec[u] = make_int4(-1, -1, -1, -1);
        return;
    }
#pragma unroll
    for (int u = 0; u < U; u++) rec[u] = ent[pick[u] != UINT32_MAX ? pick[u] : 0u];
}

__device__ __forceinline__ void wave_sync_lds() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Window edges, selection and emission for one root of a first hop with S
// windows: run [a, b) with first and last timestamps, query time t, hash key
// hp; its slots start at q * S * k.  All G lanes of the group call it
// together; my_edges is the group's row of LDS.
template <int G, int MODE, bool LAST, bool PTR, bool DIR>
__device__ __forceinline__ void multi_root(const HopArgs &p, int64_t q, int32_t x, uint32_t a, uint32_t b,
                                           float first, float last, float t, uint64_t hp, int gl,
                                           uint32_t *my_edges) {
    const uint32_t M = static_cast<uint32_t>(p.num_entries);
    const int W = p.windows;
    const int k = p.k;
    // edges i = 0..W: window s spans [edge s+1, edge s).  Bounds fall with i,
    // so edge i lies in [a, edge i-1]: edges are located four at a time, each
    // batch inside what the previous one left.  An edge that the run's first
    // and last timestamps decide is not searched.
    constexpr int NE = 4;
    uint32_t top = b;
    for (int i0 = 0; i0 <= W; i0 += NE) {
        float v[NE];
        bool act[NE];
        uint32_t c[NE];
#pragma unroll
        for (int u = 0; u < NE; u++) {
            v[u] = bound_value(t, i0 + u, p.delta);
            c[u] = a;
            act[u] = i0 + u <= W && !edge_from_summary(a, b, first, last, v[u], c[u]);
        }
        uint32_t cs[NE];
        if (PTR && b - a > HeldRun<G>::span) {      // group-uniform: long run, saved positions kept
            int ei[NE];
#pragma unroll
            for (int u = 0; u < NE; u++) ei[u] = i0 + u;
            from_pointers<G, NE>(p, x, a, b, ei, v, act, cs, gl);
        } else {
            count_below_n<G, NE, DIR>(p.tsa, M, p.tsx, p.nx, p.dir, nullptr, a, top, RunShape{a, b, first, last}, v, act, cs, gl);
        }
#pragma unroll
        for (int u = 0; u < NE; u++) {
            if (i0 + u <= W) {
                const uint32_t e = act[u] ? cs[u] : c[u];
                if (gl == 0) my_edges[i0 + u] = e;
                top = e < top ? e : top;
            }
        }
    }
    wave_sync_lds();

    const int nslots = W * k;
    const int64_t obase = q * static_cast<int64_t>(nslots);
    for (int base = 0; base < nslots; base += G) {   // group-uniform trip count
        const int e = base + gl;
        const int ee = e < nslots ? e : nslots - 1;
        const int s = ee / k;
        const int j = ee - s * k;
        const uint32_t whi = my_edges[s];
        uint32_t wlo = my_edges[s + 1];
        if (wlo > whi) wlo = whi;
        const uint32_t n = whi - wlo;
        bool has = false;
        uint32_t pick = 0;
        if constexpr (MODE == TGL_MOST_RECENT) {
            has = static_cast<uint32_t>(j) < n;
            pick = whi - 1 - static_cast<uint32_t>(j);
        } else {
            has = n > 0;
            const uint64_t key = (static_cast<uint64_t>(p.hop) << 40) |
                                 (static_cast<uint64_t>(s) << 24) | static_cast<uint64_t>(j);
            pick = wlo + static_cast<uint32_t>(__umul64hi(mix64(hp ^ key), static_cast<uint64_t>(n)));
        }
        const bool valid = e < nslots && has;
        const int4 rec = valid ? p.ent[pick] : make_int4(-1, -1, -1, -1);
        if (e < nslots) emit_slot<LAST>(p, obase + e, valid, rec, t);
    }

    if (p.o_cnt) {
        for (int w = gl; w < W; w += G) {
            const uint32_t whi = my_edges[w];
            uint32_t wlo = my_edges[w + 1];
            if (wlo > whi) wlo = whi;
            const uint32_t n = whi - wlo;
            const int32_t c = MODE == TGL_MOST_RECENT ? static_cast<int32_t>(n < static_cast<uint32_t>(k) ? n : k)
                                                      : (n > 0 ? k : 0);
            p.o_cnt[q * W + w] = c;
        }
    }
    wave_sync_lds();   // my_edges is rewritten by the group's next root
}

// First hop with more than kMultiEdges - 1 windows.  Each wavefront takes
// chunks of 64 roots:
//   phase 1, one lane per root: its time, path key and node summary are
//     packed into LDS;
//   phase 2, G lanes per root, 64 / G roots per round: the S + 1 window
//     edges, then selection and emission of the root's S * k slots.
template <int G, int MODE, bool LAST, bool PTR, bool DIR>
__global__ __launch_bounds__(kBlock) void hop_multi_wide_kernel(const HopArgs p) {
    constexpr int GPW = kWave / G;            // roots served per wavefront round
    constexpr int GPB = kBlock / G;
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const int gl = lane & (G - 1);
    const int gw = lane / G;
    __shared__ uint32_t r_a[kWavesPerBlock][kWave];
    __shared__ uint32_t r_b[kWavesPerBlock][kWave];
    __shared__ float r_f[kWavesPerBlock][kWave];
    __shared__ float r_l[kWavesPerBlock][kWave];
    __shared__ uint64_t r_hp[kWavesPerBlock][kWave];   // uniform: mix64(seedmix ^ path)
    __shared__ float r_t[kWavesPerBlock][kWave];
    __shared__ int32_t r_x[kWavesPerBlock][kWave];
    __shared__ uint32_t edges[GPB * (TGL_MAX_SNAPSHOTS + 1)];
    uint32_t *my_edges = edges + (w * GPW + gw) * (TGL_MAX_SNAPSHOTS + 1);

    const int64_t nv = p.num_roots;
    if (p.count0_out && blockIdx.x == 0 && threadIdx.x == 0) *p.count0_out = nv;
    const int64_t nchunks = (nv + kWave - 1) / kWave;

    for (int64_t c = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + w; c < nchunks;
         c += static_cast<int64_t>(gridDim.x) * kWavesPerBlock) {
        // ---- phase 1: one lane per root ----
        const int64_t v = c * kWave + lane;
        const bool valid = v < nv;
        int32_t x = -1;
        float t = 0.0f;
        if (valid) {
            x = p.rx[v];
            t = p.rt[v];
        }
        const NodeRun run = node_run(p, x, valid);
        if (valid) {
            r_a[w][lane] = run.a;
            r_b[w][lane] = run.b;
            r_f[w][lane] = run.first;
            r_l[w][lane] = run.last;
            r_hp[w][lane] = MODE == TGL_UNIFORM ? mix64(p.seedmix ^ (p.root_base + static_cast<uint64_t>(v))) : 0;
            r_t[w][lane] = t;
            r_x[w][lane] = x;
        }
        wave_sync_lds();
        // ---- phase 2: G lanes per root ----
        const int64_t rem = nv - c * kWave;
        const int nvalid = rem < kWave ? static_cast<int>(rem) : kWave;
        for (int base = 0; base < nvalid; base += GPW) {
            const int i = base + gw;
            if (i < nvalid) {                       // group-uniform
                multi_root<G, MODE, LAST, PTR, DIR>(p, c * kWave + i, r_x[w][i], r_a[w][i], r_b[w][i], r_f[w][i], r_l[w][i],
                                          r_t[w][i], r_hp[w][i], gl, my_edges);
            }
        }
        wave_sync_lds();                            // the next chunk rewrites the LDS rows
    }
}

// First hop with S > 1 windows, S + 1 <= kMultiEdges.  Each wavefront takes
// chunks of 64 roots:
//   phase 1, one lane per root: its time, path key and node summary are
//     packed into LDS;
//   phase 2, 8 lanes per root, 8 roots per round: the S + 1 window edges,
//     four at a time, each batch searched below the lowest edge found so far
//     (bounds fall with the window index), into LDS; then the per-window
//     valid counts;
//   phase 3, one lane per slot: selection, gather and emission.  Roots are
//     dense on the first hop, so a chunk's slots are one contiguous range of
//     the output and the stores coalesce.
template <int MODE, bool LAST, bool PTR, bool DIR>
__global__ __launch_bounds__(kBlock) void hop_multi_kernel(const HopArgs p) {
    constexpr int G = 8;
    constexpr int GPW = kWave / G;            // roots located per wavefront round
    constexpr int NE = 2;                     // window edges located together
    constexpr int U = 4;                      // slots per lane whose loads are in flight together
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const int gl = lane & (G - 1);
    const int gw = lane / G;
    __shared__ uint32_t r_a[kWavesPerBlock][kWave];
    __shared__ uint32_t r_b[kWavesPerBlock][kWave];
    __shared__ float r_f[kWavesPerBlock][kWave];
    __shared__ float r_l[kWavesPerBlock][kWave];
    __shared__ uint64_t r_hp[kWavesPerBlock][kWave];   // uniform: mix64(seedmix ^ path)
    __shared__ float r_t[kWavesPerBlock][kWave];
    __shared__ int32_t r_x[kWavesPerBlock][kWave];
    __shared__ uint32_t r_e[kWavesPerBlock][kWave * kMultiEdges];   // window edges of each root
    // The last hop in most-recent mode needs no lower edge for the last
    // window: its candidates are the newest entries below its upper edge,
    // and one of them is in the window exactly when its timestamp is at or
    // above the window's lower bound.  That bound is kept per root and the
    // gathered entries are checked against it instead of locating the edge.
    constexpr bool TAIL = MODE == TGL_MOST_RECENT && LAST;
    __shared__ float r_vw[kWavesPerBlock][TAIL ? kWave : 1];        // lower bound of the last window

    const uint32_t M = static_cast<uint32_t>(p.num_entries);
    const int W = p.windows;
    const int nedge = TAIL ? W : W + 1;       // window edges located per root
    const int k = p.k;
    const int nslots = W * k;                 // slots per root
    const int64_t nv = p.num_roots;
    if (p.count0_out && blockIdx.x == 0 && threadIdx.x == 0) *p.count0_out = nv;
    const int64_t nchunks = (nv + kWave - 1) / kWave;
    const uint64_t hop_key = static_cast<uint64_t>(p.hop) << 40;
    // phase 3 serves slot e = lane + 64 n of a chunk in round n: its root
    // i = e / (W k), window s and rank j (e % (W k) = s k + j) start at those
    // of e = lane and advance by the mixed-radix digits of 64 per round
    const int dj = kWave % k;
    const int ds = (kWave / k) % W;
    const int di = (kWave / k) / W;
    const int li0 = lane / nslots;
    const int ls0 = (lane - li0 * nslots) / k;
    const int lj0 = lane - li0 * nslots - ls0 * k;

    for (int64_t c = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + w; c < nchunks;
         c += static_cast<int64_t>(gridDim.x) * kWavesPerBlock) {
        // ---- phase 1: one lane per root ----
        const int64_t v = c * kWave + lane;
        const bool valid = v < nv;
        int32_t x = -1;
        float t = 0.0f;
        if (valid) {
            x = p.rx[v];
            t = p.rt[v];
        }
        const NodeRun run = node_run(p, x, valid);
        if (valid) {
            r_a[w][lane] = run.a;
            r_b[w][lane] = run.b;
            r_f[w][lane] = run.first;
            r_l[w][lane] = run.last;
            r_hp[w][lane] = MODE == TGL_UNIFORM ? mix64(p.seedmix ^ (p.root_base + static_cast<uint64_t>(v))) : 0;
            r_t[w][lane] = t;
            r_x[w][lane] = x;
            if constexpr (TAIL) r_vw[w][lane] = bound_value(t, W, p.delta);
        }
        wave_sync_lds();
        const int64_t rem = nv - c * kWave;
        const int nvalid = rem < kWave ? static_cast<int>(rem) : kWave;

        // ---- phase 2: G lanes per root locate its W + 1 window edges (W with TAIL) ----
        for (int base = 0; base < nvalid; base += GPW) {
            const int i = base + gw;
            if (i < nvalid) {                       // group-uniform
                const uint32_t a = r_a[w][i];
                const uint32_t b = r_b[w][i];
                const float first = r_f[w][i];
                const float last = r_l[w][i];
                const float ti = r_t[w][i];
                const int32_t xi = r_x[w][i];
                // a non-empty run belongs to a node inside the graph
                const int4 *rec = b > a && b - a <= TGL_NODE_INLINE ? p.nodes + static_cast<int64_t>(xi) * 8 : nullptr;
                uint32_t top = b;
                if (TAIL && gl == 0) r_e[w][i * kMultiEdges + W] = a;   // the last window reaches down to the run start
                for (int i0 = 0; i0 < nedge; i0 += NE) {
                    float vv[NE];
                    bool act[NE];
                    uint32_t cc[NE];
#pragma unroll
                    for (int u = 0; u < NE; u++) {
                        vv[u] = bound_value(ti, i0 + u, p.delta);
                        cc[u] = a;
                        act[u] = i0 + u < nedge && !edge_from_summary(a, b, first, last, vv[u], cc[u]);
                    }
                    uint32_t cs[NE];
                    if (PTR && !rec && b - a > HeldRun<G>::span) {   // group-uniform: saved positions kept
                        int ei[NE];
#pragma unroll
                        for (int u = 0; u < NE; u++) ei[u] = i0 + u;
                        from_pointers<G, NE>(p, xi, a, b, ei, vv, act, cs, gl);
                    } else {
                        count_below_n<G, NE, DIR>(p.tsa, M, p.tsx, p.nx, p.dir, rec, a, top, RunShape{a, b, first, last}, vv,
                                             act, cs, gl);
                    }
#pragma unroll
                    for (int u = 0; u < NE; u++) {
                        if (i0 + u < nedge) {
                            const uint32_t e = act[u] ? cs[u] : cc[u];
                            if (gl == 0) r_e[w][i * kMultiEdges + i0 + u] = e;
                            top = e < top ? e : top;
                        }
                    }
                }
            }
        }
        wave_sync_lds();
        // valid slots per (root, window) group, for the next hop
        if (p.o_cnt) {
            for (int g = lane; g < nvalid * W; g += kWave) {
                const int i = g / W;
                const int s = g - i * W;
                const uint32_t whi = r_e[w][i * kMultiEdges + s];
                const uint32_t wlo = r_e[w][i * kMultiEdges + s + 1];
                const uint32_t n = wlo < whi ? whi - wlo : 0u;
                p.o_cnt[(c * kWave + i) * W + s] = MODE == TGL_MOST_RECENT
                                                       ? static_cast<int32_t>(n < static_cast<uint32_t>(k) ? n : k)
                                                       : (n > 0 ? k : 0);
            }
        }

        // ---- phase 3: one lane per slot ----
        const int total = nvalid * nslots;
        const int64_t obase = c * kWave * static_cast<int64_t>(nslots);
        OutRow orow{p.o_nbr + obase, p.o_eid + obase, p.o_ts + obase, p.o_dt + obase, nullptr};
        if constexpr (!LAST) orow.first = p.o_first ? p.o_first + obase : nullptr;
        int ci = li0, cs = ls0, cj = lj0;           // (i, s, j) of this lane's slot in the round
        for (int e0 = 0; e0 < total; e0 += U * kWave) {
            uint32_t pick[U];                       // UINT32_MAX: PAD slot
            int iu[U];
            bool tail[U];                           // TAIL: a slot of the last window
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int e = e0 + u * kWave + lane;
                const bool act = e < total;
                const int i = act ? ci : 0;
                const int s = act ? cs : 0;
                const int j = cj;
                iu[u] = i;
                tail[u] = TAIL && s == W - 1;
                cj += dj;
                cs += ds;
                ci += di;
                if (cj >= k) {
                    cj -= k;
                    cs += 1;
                }
                if (cs >= W) {
                    cs -= W;
                    ci += 1;
                }
                const uint32_t whi = r_e[w][i * kMultiEdges + s];
                uint32_t wlo = r_e[w][i * kMultiEdges + s + 1];
                if (wlo > whi) wlo = whi;
                const uint32_t n = whi - wlo;
                if constexpr (MODE == TGL_MOST_RECENT) {
                    pick[u] = act && static_cast<uint32_t>(j) < n ? whi - 1 - static_cast<uint32_t>(j) : UINT32_MAX;
                } else {
                    const uint64_t key = hop_key | (static_cast<uint64_t>(s) << 24) | static_cast<uint64_t>(j);
                    pick[u] = act && n > 0
                                  ? wlo + static_cast<uint32_t>(__umul64hi(mix64(r_hp[w][i] ^ key), static_cast<uint64_t>(n)))
                                  : UINT32_MAX;
                }
            }
            int4 rec[U];
            gather_records<U>(p.ent, static_cast<uint32_t>(p.num_entries), pick, rec);
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int e = e0 + u * kWave + lane;
                bool valid = pick[u] != UINT32_MAX;
                if constexpr (TAIL) valid = valid && (!tail[u] || __int_as_float(rec[u].y) >= r_vw[w][iu[u]]);
                if (e < total) emit_at<LAST>(orow, static_cast<uint32_t>(e), valid, rec[u], r_t[w][iu[u]]);
            }
        }
        wave_sync_lds();                            // the next chunk rewrites the LDS rows
    }
}

// Window [lo, hi) of a root with run [a, b) between the float thresholds
// vl <= ts < vh (one window per root), by the G lanes of its group.  An edge
// that the run's first and last timestamps decide is not searched.  NB is
// the number of window edges: 1 when windows are unbounded below (lo = a),
// else 2.
template <int G, int NB, bool PTR, bool DIR>
__device__ __forceinline__ void locate_window(const HopArgs &p, int32_t x, uint32_t a, uint32_t b, float first,
                                              float last, float vh, float vl, int gl, uint32_t &lo, uint32_t &hi) {
    const uint32_t M = static_cast<uint32_t>(p.num_entries);
    // a non-empty run belongs to a node inside the graph
    const int4 *rec = b > a && b - a <= TGL_NODE_INLINE ? p.nodes + static_cast<int64_t>(x) * 8 : nullptr;
    float v[NB];
    bool act[NB];
    uint32_t c[NB];
#pragma unroll
    for (int i = 0; i < NB; i++) {
        v[i] = i == 0 ? vh : vl;
        c[i] = a;
        act[i] = !edge_from_summary(a, b, first, last, v[i], c[i]);
    }
    uint32_t cs[NB];
    if (PTR && !rec && b - a > HeldRun<G>::span) {       // group-uniform: hop 1, saved positions kept
        int ei[NB];
#pragma unroll
        for (int i = 0; i < NB; i++) ei[i] = i;             // hop 1 with one window: edges t and t - D
        from_pointers<G, NB>(p, x, a, b, ei, v, act, cs, gl);
    } else {
        count_below_n<G, NB, DIR>(p.tsa, M, p.tsx, p.nx, p.dir, rec, a, b, RunShape{a, b, first, last}, v, act, cs, gl);
    }
    hi = act[0] ? cs[0] : c[0];
    lo = NB == 1 ? a : (act[NB - 1] ? cs[NB - 1] : c[NB - 1]);
    if (lo > hi) lo = hi;
}

// One hop with one window per root (every hop except a first hop with several
// snapshots).  Each wavefront takes chunks of 64 candidate roots:
//   phase 1, one lane per candidate: hop 1 takes root v as given; later hops
//     take slot v of the previous hop, valid when its nbr >= 0, as the root
//     with index off(g) + j for g = v / k_prev, j = v % k_prev, off the
//     exclusive scan of the previous hop's group counts (and write its parent
//     index).  Every lane loads its root's time and run bounds, except a root
//     whose entry carried the neighbour-first hint (its window is empty); the
//     valid roots are packed, in order, into LDS;
//   phase 2, G lanes per root, 64 / G roots per round: the window [lo, hi);
//   phase 3, one lane per slot: selection, gather and emit.  The packed roots
//     have consecutive indices, so the slots of a chunk are one contiguous
//     range of the output and the stores coalesce.
// WIN (one window unbounded below, a T-CSR with neighbour histories): the
// window of a root of hop >= 2 is the history of the entry it came from,
// which the previous hop gathered with the entry; phase 1 takes it from
// there, and reads no node record and leaves nothing to search.  A hop that
// is not the last gathers the histories of its picks for the next hop.
// DIR (a T-CSR with time directories): phase 2 starts the search of a long
// run from its directory.
template <int G, int MODE, bool LAST, bool FIRST, int NB, bool PTR, bool WIN, bool DIR>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(WIN && !FIRST ? 4 : (NB == 1 ? 7 : 6)))) void hop_single_kernel(const HopArgs p) {
    static_assert(FIRST || !PTR, "saved window edges are kept for hop 1 only");
    static_assert(!(PTR && DIR), "saved window edges replace the directory");
    static_assert(!WIN || NB == 1, "histories give windows unbounded below");
    constexpr int GPW = kWave / G;            // roots located per wavefront round
    // slots per lane whose loads are in flight together.  A hop that takes its
    // windows from the histories searches nothing, and its registers go to
    // ten record loads per lane: a chunk of 64 roots with k = 10 then issues
    // all its gathers at once (4 waves per SIMD instead of 8)
    constexpr int U = WIN && !FIRST ? 10 : 4;
    const int lane = lane_id();
    const int w = threadIdx.x / kWave;
    const int gl = lane & (G - 1);
    const int gw = lane / G;
    __shared__ uint32_t r_lo[kWavesPerBlock][kWave];   // run start, then window start
    __shared__ uint32_t r_n[kWavesPerBlock][kWave];    // run end, then window size
    __shared__ float r_f[kWavesPerBlock][kWave];       // first and last timestamp of the run
    __shared__ float r_l[kWavesPerBlock][kWave];
    __shared__ int64_t r_q0[kWavesPerBlock];           // index of the first packed root
    // uniform: mix64(seedmix ^ path) ^ (hop << 40 | s << 24), so that the
    // draw of rank j hashes it ^ j (the key fields do not overlap)
    __shared__ uint64_t r_hp[kWavesPerBlock][kWave];
    __shared__ float r_t[kWavesPerBlock][kWave];
    __shared__ int32_t r_x[kWavesPerBlock][kWave];     // node of each packed root
    __shared__ float r_vh[kWavesPerBlock][kWave];      // window thresholds: vl <= ts < vh
    __shared__ float r_vl[kWavesPerBlock][NB == 2 ? kWave : 1];
    __shared__ uint8_t r_need[kWavesPerBlock][kWave];  // packed roots whose window needs a search

    const int64_t pk = FIRST ? 1 : p.p_k;
    int64_t nv;
    if constexpr (FIRST) {
        nv = p.num_roots;
        if (p.count0_out && blockIdx.x == 0 && threadIdx.x == 0) *p.count0_out = nv;
    } else {
        const int64_t groups = p.p_groups_dyn ? *p.p_groups_dyn : p.p_groups_static;
        nv = groups * pk;
    }
    const int64_t nchunks = (nv + kWave - 1) / kWave;
    const uint64_t S = static_cast<uint64_t>(p.S);
    const uint64_t path1 = p.root_base * S * static_cast<uint64_t>(pk);   // hop-1 children: + v
    const int k = p.k;
    const uint64_t hop_key = static_cast<uint64_t>(p.hop) << 40;
    // phase 3 serves slot e = lane + 64 n of a chunk in round n: its root
    // e / k and rank e % k start at (lane / k, lane % k) and advance by
    // (64 / k, 64 % k) per round, with a carry
    const int di = kWave / k;
    const int dj = kWave - di * k;
    const int li0 = lane / k;
    const int lj0 = lane - li0 * k;

    for (int64_t c = static_cast<int64_t>(blockIdx.x) * kWavesPerBlock + w; c < nchunks;
         c += static_cast<int64_t>(gridDim.x) * kWavesPerBlock) {
        // ---- phase 1: one lane per candidate root ----
        const int64_t v = c * kWave + lane;
        bool valid;
        int32_t x = -1;
        float t = 0.0f;
        int64_t q = 0;
        int32_t s = 0;
        uint64_t path = 0;
        float ta = 0.0f;                        // the time the windows are placed at
        if constexpr (FIRST) {
            valid = v < nv;
            if (valid) {
                x = p.rx[v];
                t = p.rt[v];
                ta = t;
                q = v;
                path = p.root_base + static_cast<uint64_t>(v);
            }
        } else {
            x = v < nv ? p.p_nbr[v] : -1;
            valid = x >= 0;
            if (valid) {
                t = p.p_ts[v];
                ta = t;
                const int64_t g = v / pk;
                const int64_t j = v - g * pk;
                q = p.p_tile[g / kScanTile] + p.p_local[g] + j;
                if (p.p_s) {
                    s = p.p_s[g];
                    path = p.p_path[g] * static_cast<uint64_t>(pk) + static_cast<uint64_t>(j);
                } else {
                    s = static_cast<int32_t>(static_cast<uint64_t>(g) % S);
                    path = path1 + static_cast<uint64_t>(v);
                }
                if (p.anchor == TGL_ANCHOR_ROOT) {
                    // hop-1 ancestor: hop-2 roots come from hop-1 group (r, s) = g
                    ta = p.p_t0 ? p.p_t0[g] : p.rt[static_cast<uint64_t>(g) / S];
                    if (p.o_t0) p.o_t0[q] = ta;
                }
                p.o_parent[q] = v;
                if (p.o_s) {
                    p.o_s[q] = s;
                    p.o_path[q] = path;
                }
            }
        }
        NodeRun run{0u, 0u, 0.0f, 0.0f};
        float vh = 0.0f, vl = 0.0f;
        uint32_t lo = 0, hi = 0;
        bool need = false;
        if constexpr (WIN && !FIRST) {
            // the window is the history of the entry this root came from,
            // clamped into the entries
            if (valid) {
                const uint2 wv = p.p_win[v];
                const uint32_t M = static_cast<uint32_t>(p.num_entries);
                hi = wv.y < M ? wv.y : M;
                lo = wv.x < hi ? wv.x : hi;
            }
        } else {
            // a root whose entry carried the hint has an empty window: its node
            // record is not read
            bool known_empty = false;
            if constexpr (!FIRST) known_empty = valid && p.p_first && p.p_first[v] != 0;
            run = node_run(p, x, valid && !known_empty);
            // window thresholds; with the root anchor the window also ends below t
            vh = bound_value(ta, s, p.delta);
            if (p.anchor == TGL_ANCHOR_ROOT && t < vh) vh = t;
            if constexpr (NB == 2) vl = bound_value(ta, s + 1, p.delta);
            // window edges the run's first and last timestamps decide
            lo = run.a;
            hi = run.a;
            if (valid) {
                need = !edge_from_summary(run.a, run.b, run.first, run.last, vh, hi);
                if constexpr (NB == 2) need |= !edge_from_summary(run.a, run.b, run.first, run.last, vl, lo);
                if (lo > hi) lo = hi;
            }
        }
        const uint64_t mask = __ballot(valid);
        const uint64_t need_mask = __ballot(valid && need);
        if (valid) {
            const int r = rank_below(mask);
            r_lo[w][r] = need ? run.a : lo;
            r_n[w][r] = need ? run.b : hi - lo;
            if (r == 0) r_q0[w] = q;             // packed roots are q0, q0 + 1, ...
            r_hp[w][r] = MODE == TGL_UNIFORM
                             ? mix64(p.seedmix ^ path) ^ hop_key ^ (static_cast<uint64_t>(static_cast<uint32_t>(s)) << 24)
                             : 0;
            r_t[w][r] = t;
            if constexpr (!(WIN && !FIRST)) {
                r_f[w][r] = run.first;
                r_l[w][r] = run.last;
                r_x[w][r] = x;
                r_vh[w][r] = vh;
                if constexpr (NB == 2) r_vl[w][r] = vl;
                if (need) r_need[w][rank_below(need_mask)] = static_cast<uint8_t>(r);
            }
            if (!need && p.o_cnt) {
                const uint32_t n = hi - lo;
                p.o_cnt[q] = MODE == TGL_MOST_RECENT ? static_cast<int32_t>(n < static_cast<uint32_t>(k) ? n : k)
                                                     : (n > 0 ? k : 0);
            }
        }
        wave_sync_lds();
        const int nvalid = __popcll(mask);
        const int nneed = __popcll(need_mask);

        // ---- phase 2: G lanes per root search the windows phase 1 left open ----
        for (int base = 0; base < (WIN && !FIRST ? 0 : nneed); base += GPW) {
            if (base + gw < nneed) {                // group-uniform
                const int i = r_need[w][base + gw];
                uint32_t wlo, whi;
                locate_window<G, NB, PTR, DIR>(p, r_x[w][i], r_lo[w][i], r_n[w][i], r_f[w][i], r_l[w][i], r_vh[w][i],
                                          NB == 2 ? r_vl[w][i] : 0.0f, gl, wlo, whi);
                if (gl == 0) {
                    r_lo[w][i] = wlo;
                    r_n[w][i] = whi - wlo;
                    if (p.o_cnt) {
                        const uint32_t n = whi - wlo;
                        p.o_cnt[r_q0[w] + i] = MODE == TGL_MOST_RECENT
                                                 ? static_cast<int32_t>(n < static_cast<uint32_t>(k) ? n : k)
                                                 : (n > 0 ? k : 0);
                    }
                }
            }
        }
        wave_sync_lds();

        // ---- phase 3: one lane per slot ----
        // slot e of the chunk (root i = e / k, rank j = e % k) is output
        // q0 * k + e, packed roots having consecutive indices
        const int total = nvalid * k;
        const int64_t obase = total > 0 ? uniform64(r_q0[w]) * k : 0;
        OutRow orow{p.o_nbr + obase, p.o_eid + obase, p.o_ts + obase, p.o_dt + obase, nullptr, nullptr};
        if constexpr (!LAST && !WIN) orow.first = p.o_first ? p.o_first + obase : nullptr;
        if constexpr (!LAST && WIN) orow.win = p.o_win + obase;
        int ci = li0, cj = lj0;                     // (i, j) of this lane's slot in the round
        for (int e0 = 0; e0 < total; e0 += U * kWave) {
            uint32_t pick[U];                       // UINT32_MAX: PAD slot
            int iu[U];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int e = e0 + u * kWave + lane;
                const bool act = e < total;
                const int i = act ? ci : 0;
                const int j = cj;
                iu[u] = i;
                cj += dj;
                ci += di;
                if (cj >= k) {
                    cj -= k;
                    ci += 1;
                }
                const uint32_t lo = r_lo[w][i];
                const uint32_t n = r_n[w][i];
                if constexpr (MODE == TGL_MOST_RECENT) {
                    pick[u] = act && static_cast<uint32_t>(j) < n ? lo + n - 1 - static_cast<uint32_t>(j) : UINT32_MAX;
                } else {
                    pick[u] = act && n > 0
                                  ? lo + static_cast<uint32_t>(__umul64hi(mix64(r_hp[w][i] ^ static_cast<uint64_t>(j)),
                                                                          static_cast<uint64_t>(n)))
                                  : UINT32_MAX;
                }
            }
            int4 rec[U];
            if constexpr (WIN && !LAST) {
                // the histories are loaded once the entries are in: a pick whose
                // entry carries the neighbour-first hint has an empty history,
                // and reads entry 0's (one cached line) instead of its own
                gather_records<U>(p.ent, static_cast<uint32_t>(p.num_entries), pick, rec);
                uint2 hv[U];
#pragma unroll
                for (int u = 0; u < U; u++)
                    hv[u] = p.hist[pick[u] != UINT32_MAX && rec[u].x >= 0 ? pick[u] : 0u];
#pragma unroll
                for (int u = 0; u < U; u++) {
                    const int e = e0 + u * kWave + lane;
                    if (e < total && pick[u] != UINT32_MAX) orow.win[e] = rec[u].x >= 0 ? hv[u] : make_uint2(0u, 0u);
                }
            } else {
                gather_records<U>(p.ent, static_cast<uint32_t>(p.num_entries), pick, rec);
            }
#pragma unroll
            for (int u = 0; u < U; u++) {
                const int e = e0 + u * kWave + lane;
                if (e < total) emit_at<LAST>(orow, static_cast<uint32_t>(e), pick[u] != UINT32_MAX, rec[u], r_t[w][iu[u]]);
            }
        }
        wave_sync_lds();                            // the next chunk rewrites the LDS rows
    }
}

template <int MODE, bool LAST>
void launch_mode_last(int G, bool first, bool multi, bool win, const HopArgs &a, int64_t work, hipStream_t st) {
    // `work` candidate roots (hop 1: roots; later hops: previous slots), 64 per wavefront
    int64_t blocks = (work + kBlock - 1) / kBlock;
    if (blocks < 1) blocks = 1;
    if (blocks > kMaxGrid) blocks = kMaxGrid;
    const unsigned nb = static_cast<unsigned>(blocks);
    // kernels that search long runs start from the time directories when the
    // T-CSR has them; those that keep saved window edges search from those
    const bool dir = a.dir != nullptr;
    if (multi && a.windows + 1 <= kMultiEdges) {   // first hop only
        if (a.ptr) hop_multi_kernel<MODE, LAST, true, false><<<nb, kBlock, 0, st>>>(a);
        else if (dir) hop_multi_kernel<MODE, LAST, false, true><<<nb, kBlock, 0, st>>>(a);
        else hop_multi_kernel<MODE, LAST, false, false><<<nb, kBlock, 0, st>>>(a);
    } else if (multi && a.ptr) {              // first hop only; saved window edges kept
        switch (G) {
            case 16: hop_multi_wide_kernel<16, MODE, LAST, true, false><<<nb, kBlock, 0, st>>>(a); break;
            case 32: hop_multi_wide_kernel<32, MODE, LAST, true, false><<<nb, kBlock, 0, st>>>(a); break;
            default: hop_multi_wide_kernel<64, MODE, LAST, true, false><<<nb, kBlock, 0, st>>>(a); break;
        }
    } else if (multi && dir) {                // first hop only
        switch (G) {
            case 16: hop_multi_wide_kernel<16, MODE, LAST, false, true><<<nb, kBlock, 0, st>>>(a); break;
            case 32: hop_multi_wide_kernel<32, MODE, LAST, false, true><<<nb, kBlock, 0, st>>>(a); break;
            default: hop_multi_wide_kernel<64, MODE, LAST, false, true><<<nb, kBlock, 0, st>>>(a); break;
        }
    } else if (multi) {                       // first hop only
        switch (G) {
            case 16: hop_multi_wide_kernel<16, MODE, LAST, false, false><<<nb, kBlock, 0, st>>>(a); break;
            case 32: hop_multi_wide_kernel<32, MODE, LAST, false, false><<<nb, kBlock, 0, st>>>(a); break;
            default: hop_multi_wide_kernel<64, MODE, LAST, false, false><<<nb, kBlock, 0, st>>>(a); break;
        }
    } else {
        // the window search uses 8 lanes per root whatever the fanout; one
        // window edge when windows are unbounded below, else two
        const bool ptr = first && a.ptr;
        if (win) {                            // windows unbounded below, neighbour histories kept
            if (ptr) hop_single_kernel<8, MODE, LAST, true, 1, true, true, false><<<nb, kBlock, 0, st>>>(a);
            else if (first && dir) hop_single_kernel<8, MODE, LAST, true, 1, false, true, true><<<nb, kBlock, 0, st>>>(a);
            else if (first) hop_single_kernel<8, MODE, LAST, true, 1, false, true, false><<<nb, kBlock, 0, st>>>(a);
            else hop_single_kernel<8, MODE, LAST, false, 1, false, true, false><<<nb, kBlock, 0, st>>>(a);
        } else if (a.delta_inf) {
            if (ptr) hop_single_kernel<8, MODE, LAST, true, 1, true, false, false><<<nb, kBlock, 0, st>>>(a);
            else if (first && dir) hop_single_kernel<8, MODE, LAST, true, 1, false, false, true><<<nb, kBlock, 0, st>>>(a);
            else if (first) hop_single_kernel<8, MODE, LAST, true, 1, false, false, false><<<nb, kBlock, 0, st>>>(a);
            else if (dir) hop_single_kernel<8, MODE, LAST, false, 1, false, false, true><<<nb, kBlock, 0, st>>>(a);
            else hop_single_kernel<8, MODE, LAST, false, 1, false, false, false><<<nb, kBlock, 0, st>>>(a);
        } else {
            if (ptr) hop_single_kernel<8, MODE, LAST, true, 2, true, false, false><<<nb, kBlock, 0, st>>>(a);
            else if (first && dir) hop_single_kernel<8, MODE, LAST, true, 2, false, false, true><<<nb, kBlock, 0, st>>>(a);
            else if (first) hop_single_kernel<8, MODE, LAST, true, 2, false, false, false><<<nb, kBlock, 0, st>>>(a);
            else if (dir) hop_single_kernel<8, MODE, LAST, false, 2, false, false, true><<<nb, kBlock, 0, st>>>(a);
            else hop_single_kernel<8, MODE, LAST, false, 2, false, false, false><<<nb, kBlock, 0, st>>>(a);
        }
    }
}

void launch_hop(int G, int mode, bool first, bool multi, bool last, bool win, const HopArgs &a, int64_t work,
                hipStream_t st) {
    if (mode == TGL_MOST_RECENT) {
        last ? launch_mode_last<TGL_MOST_RECENT, true>(G, first, multi, win, a, work, st)
             : launch_mode_last<TGL_MOST_RECENT, false>(G, first, multi, win, a, work, st);
    } else {
        last ? launch_mode_last<TGL_UNIFORM, true>(G, first, multi, win, a, work, st)
             : launch_mode_last<TGL_UNIFORM, false>(G, first, multi, win, a, work, st);
    }
}

// lanes per root for first hops with several windows: the slot count rounded
// up to a power of two, in [16, 64]
int pick_group(int64_t slots_per_root) {
    int g = 16;
    while (g < 64 && g < slots_per_root) g <<= 1;
    return g;
}

// Saved window edges at the start of every run: pointers[i * N + x] = indptr[x]
// (clamped into [0, M]).
__global__ __launch_bounds__(kBlock) void pointers_reset_kernel(const int64_t *__restrict__ indptr, int64_t N,
                                                                 int64_t M, int64_t n, uint32_t *__restrict__ ptr) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    for (int64_t e = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; e < n; e += stride) {
        const int64_t x = e % N;
        int64_t a = indptr[x];
        a = a < 0 ? 0 : (a > M ? M : a);
        ptr[e] = static_cast<uint32_t>(a);
    }
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

// Exclusive scan of a hop's per-group valid counts, first pass, tiles of
// kScanTile groups per block: the counts are overwritten with each group's
// offset within its tile, and the tile totals go to tile_off (which
// launch_scan_partials then turns into exclusive tile offsets, writing the
// grand total, the next hop's root count).  The next hop's index of group
// g's slot j is tile_off[g / kScanTile] + cnt[g] + j.  Against a reduce pass
// and an apply pass, this reads the counts once and writes 4 bytes per group
// instead of 8.
__global__ __launch_bounds__(kBlock) void group_scan_kernel(int32_t *__restrict__ cnt, int64_t n_static,
                                                            const int64_t *__restrict__ n_dyn,
                                                            int64_t *__restrict__ tile_off) {
    __shared__ int64_t lds[kBlock / kWave];
    const int64_t n = n_dyn ? *n_dyn : n_static;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kScanTile + static_cast<int64_t>(threadIdx.x) * kScanItems;
    int32_t v[kScanItems];
    int64_t sum = 0;
#pragma unroll
    for (int i = 0; i < kScanItems; i++) {
        const int64_t idx = base + i;
        v[i] = idx < n ? cnt[idx] : 0;
        sum += v[i];
    }
    int64_t total;
    int64_t run = block_exclusive_sum<int64_t>(sum, lds, &total);
#pragma unroll
    for (int i = 0; i < kScanItems; i++) {
        const int64_t idx = base + i;
        if (idx < n) cnt[idx] = static_cast<int32_t>(run);        // < kScanTile * TGL_MAX_FANOUT
        run += v[i];
    }
    if (threadIdx.x == 0) tile_off[blockIdx.x] = total;
}

struct SampleWs {
    // valid slots per group of hop h, then their offsets in the scan tile:
    // hop h writes cnt[h & 1] while it reads hop h - 1's offsets from
    // cnt[(h - 1) & 1] (a single buffer would let a later chunk read a count
    // that an earlier chunk of the same launch has just written)
    int32_t *cnt[2] = {nullptr, nullptr};
    int64_t *tile_off = nullptr;     // per scan tile: total, then exclusive offset
    int32_t *s[2] = {nullptr, nullptr};       // window per root (hops 2..L-1)
    uint64_t *path[2] = {nullptr, nullptr};   // path per root (hops 2..L-1)
    float *t0[2] = {nullptr, nullptr};        // hop-1 ancestor time per root (hops 2..L-1, root anchor)
    uint8_t *first[2] = {nullptr, nullptr};   // TGL_NBR_FIRST hint per slot (hops 1..L-1) ...
    uint2 *win[2] = {nullptr, nullptr};       // ... or, in the same memory, the next hop's windows
    size_t bytes = 0;
};

// Workspace: per-group counts and offsets for the largest hop h < L (two
// alternating buffers when L >= 3: hop h writes buffer h & 1, hop h + 1 reads
// it) and scan partials; window, path and hop-1 ancestor time of the roots of
// hops 2..L-1 (two alternating buffers); per slot of hops 1..L-1 the
// neighbour-first hint, or with one snapshot room for the history span of the
// slot's entry (hop h writes buffer h & 1, hop h + 1 reads it).
SampleWs carve_sample_ws(void *base, int32_t hops, const int64_t *cap, int32_t S) {
    SampleWs w;
    Carver cv(base);
    if (hops >= 2) {
        int64_t max_slots = 0;                 // slots of hops 1..L-1
        for (int h = 1; h < hops; h++) max_slots = cap[h] > max_slots ? cap[h] : max_slots;
        const int nfirst = hops >= 3 ? 2 : 1;
        // a slot carries a hint byte, or with one snapshot the history span of
        // its entry (when the T-CSR has them)
        const size_t per_slot = S == 1 ? sizeof(uint2) : 1;
        for (int i = 0; i < nfirst; i++) {
            uint8_t *b = cv.take<uint8_t>(static_cast<size_t>(max_slots) * per_slot);
            w.first[(1 + i) & 1] = b;
            w.win[(1 + i) & 1] = reinterpret_cast<uint2 *>(b);
        }
        int64_t max_groups = cap[0] * S;      // hop-1 groups
        for (int h = 2; h < hops; h++) max_groups = cap[h - 1] > max_groups ? cap[h - 1] : max_groups;
        const int ncnt = hops >= 3 ? 2 : 1;
        for (int i = 0; i < ncnt; i++) w.cnt[(1 + i) & 1] = cv.take<int32_t>(static_cast<size_t>(max_groups));
        w.tile_off = cv.take<int64_t>(static_cast<size_t>(scan_tiles(max_groups) + 1));
        if (hops >= 3) {
            int64_t max_mid = 0;               // roots of hops 2..L-1
            for (int h = 2; h < hops; h++) max_mid = cap[h - 1] > max_mid ? cap[h - 1] : max_mid;
            const int nbuf = hops >= 4 ? 2 : 1;
            for (int i = 0; i < nbuf; i++) {
                w.s[i] = cv.take<int32_t>(static_cast<size_t>(max_mid));
                w.path[i] = cv.take<uint64_t>(static_cast<size_t>(max_mid));
                w.t0[i] = cv.take<float>(static_cast<size_t>(max_mid));
            }
        }
    }
    w.bytes = cv.size();
    if (w.bytes == 0) w.bytes = 256;
    return w;
}

// Workspace of tgl_sample_noalloc: a fixed area of device memory that the
// code object holds on every GPU it is loaded on, for callers that cannot
// allocate.  Host code never uses the array's name as an address: its
// device address is looked up once per device and kept in scratch_dev.
// Every call on one GPU shares that GPU's area.
static __device__ __align__(256) uint8_t scratch[TGL_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
void *scratch_dev[kMaxDevices] = {};
std::mutex scratch_mu;

// The device address of `scratch` on the current device, looked up on the
// first call there.
tgl_status scratch_ptr(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TGL_EDEVICE;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_dev[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return TGL_EDEVICE;
        scratch_dev[dev] = ptr;
    }
    *out = scratch_dev[dev];
    return TGL_OK;
}

// Host-side argument checks of tgl_sample_ex (nothing is enqueued on
// failure); fills cap with the per-hop capacities.
tgl_status sample_check(const tgl_tcsr *g, const int32_t *roots, const float *root_ts, int64_t num_roots,
                        int32_t hops, const int32_t *fanouts, int32_t mode, int32_t num_snapshots,
                        float snapshot_len, const tgl_sample_opts *opts, const tgl_hop_out *outs,
                        const int64_t *counts, int64_t *cap) {
    if (!g || !outs || !counts) return TGL_EINVAL;
    const int32_t anchor = opts ? opts->anchor : TGL_ANCHOR_OWN;
    if (anchor != TGL_ANCHOR_OWN && anchor != TGL_ANCHOR_ROOT) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(opts ? opts->pointers : nullptr) & 3u) != 0) return TGL_EINVAL;
    if (!sample_args_ok(num_roots, hops, fanouts, num_snapshots)) return TGL_EINVAL;
    if (mode != TGL_MOST_RECENT && mode != TGL_UNIFORM) return TGL_EINVAL;
    if (snapshot_len != snapshot_len || !(snapshot_len > 0.0f)) return TGL_EINVAL;
    if (__builtin_isinf(snapshot_len) && num_snapshots != 1) return TGL_EINVAL;
    if (g->num_nodes < 1 || g->num_nodes > INT32_MAX) return TGL_EINVAL;
    if (g->num_entries < 0 || g->num_entries > static_cast<int64_t>(UINT32_MAX)) return TGL_EINVAL;
    if (!g->indptr || (g->num_entries > 0 && !g->entries)) return TGL_EINVAL;
    if (g->num_entries > 0 && !g->ts) return TGL_EINVAL;
    if (!g->nodes || (reinterpret_cast<uintptr_t>(g->nodes) & 127u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(g->entries) & 15u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(g->ts) & 15u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(g->ts_index) & 15u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(g->hist) & 7u) != 0) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(g->dir) & 7u) != 0) return TGL_EINVAL;
    if (num_roots > 0 && (!roots || !root_ts)) return TGL_EINVAL;
    if (!capacities(num_roots, hops, fanouts, num_snapshots, cap)) return TGL_EINVAL;
    for (int h = 0; h < hops; h++) {
        const tgl_hop_out &o = outs[h];
        if (cap[h + 1] > 0 && (!o.nbr || !o.eid || !o.ts || !o.dt)) return TGL_EINVAL;
        if (h > 0 && cap[h] > 0 && !o.parent) return TGL_EINVAL;
    }
    return TGL_OK;
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

tgl_status tgl_sample_ex(const tgl_tcsr *g, const int32_t *roots, const float *root_ts,
                         int64_t num_roots, int32_t hops, const int32_t *fanouts, int32_t mode,
                         int32_t num_snapshots, float snapshot_len, uint64_t seed,
                         uint64_t root_base, const tgl_sample_opts *opts, const tgl_hop_out *outs,
                         int64_t *counts, void *workspace, size_t workspace_bytes, void *stream) {
    // ---- host-side argument checks (nothing is enqueued on failure) ----
    int64_t cap[TGL_MAX_HOPS + 1];
    const tgl_status chk = sample_check(g, roots, root_ts, num_roots, hops, fanouts, mode, num_snapshots,
                                        snapshot_len, opts, outs, counts, cap);
    if (chk != TGL_OK) return chk;
    const int32_t anchor = opts ? opts->anchor : TGL_ANCHOR_OWN;
    uint32_t *const pointers = opts ? opts->pointers : nullptr;
    const bool dinf = __builtin_isinf(snapshot_len);
    const SampleWs need = carve_sample_ws(nullptr, hops, cap, num_snapshots);
    if (hops >= 2 && (!workspace || workspace_bytes < need.bytes)) return TGL_ENOSPACE;
    const SampleWs ws = carve_sample_ws(workspace, hops, cap, num_snapshots);

    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();   // clear a stale error so launch checks are ours

    HopArgs a{};
    a.indptr = g->indptr;
    a.ent = reinterpret_cast<const int4 *>(g->entries);
    a.tsa = g->ts;
    a.tsx = g->num_entries > 0 ? g->ts_index : nullptr;
    a.nx = static_cast<uint32_t>(tgl_index_len(g->num_entries));
    a.nodes = reinterpret_cast<const int4 *>(g->nodes);
    a.dir = g->num_entries > 0 ? reinterpret_cast<const uint2 *>(g->dir) : nullptr;
    // windows of hops >= 2 from the histories of the previous hop's entries:
    // one snapshot unbounded below (either anchor then places the window of
    // a root below its own time)
    const bool win = g->hist && g->num_entries > 0 && num_snapshots == 1 && dinf && hops >= 2;
    a.hist = win ? reinterpret_cast<const uint2 *>(g->hist) : nullptr;
    a.num_nodes = g->num_nodes;
    a.num_entries = g->num_entries;
    a.rx = roots;
    a.rt = root_ts;
    a.num_roots = num_roots;
    a.root_base = root_base;
    a.S = num_snapshots;
    a.delta = snapshot_len;
    a.delta_inf = dinf ? 1 : 0;
    a.anchor = anchor;
    a.seedmix = mix64(seed ^ kGolden);

    const int32_t S = num_snapshots;
    for (int h = 1; h <= hops; h++) {
        const bool last = h == hops;
        const int32_t k = fanouts[h - 1];
        const tgl_hop_out &o = outs[h - 1];
        a.hop = h;
        a.k = k;
        a.ptr = h == 1 ? pointers : nullptr;
        a.windows = h == 1 ? S : 1;
        a.o_nbr = o.nbr;
        a.o_eid = o.eid;
        a.o_ts = o.ts;
        a.o_dt = o.dt;
        a.o_parent = h >= 2 ? o.parent : nullptr;
        a.o_cnt = last ? nullptr : ws.cnt[h & 1];
        // window and path of this hop's roots are kept for hop h + 1 (hop-1
        // children derive them from their slot index instead)
        const bool keep = h >= 2 && h < hops;
        a.o_s = keep ? ws.s[h & 1] : nullptr;
        a.o_path = keep ? ws.path[h & 1] : nullptr;
        a.o_t0 = keep && anchor == TGL_ANCHOR_ROOT ? ws.t0[h & 1] : nullptr;
        a.o_first = last || win ? nullptr : ws.first[h & 1];
        a.p_first = h >= 2 && !win ? ws.first[(h - 1) & 1] : nullptr;
        a.o_win = !last && win ? ws.win[h & 1] : nullptr;
        a.p_win = h >= 2 && win ? ws.win[(h - 1) & 1] : nullptr;
        a.count0_out = h == 1 ? counts : nullptr;
        if (h >= 2) {
            const tgl_hop_out &po = outs[h - 2];
            a.p_nbr = po.nbr;
            a.p_ts = po.ts;
            a.p_local = ws.cnt[(h - 1) & 1];
            a.p_tile = ws.tile_off;
            a.p_k = fanouts[h - 2];
            a.p_s = h >= 3 ? ws.s[(h - 1) & 1] : nullptr;
            a.p_path = h >= 3 ? ws.path[(h - 1) & 1] : nullptr;
            a.p_t0 = h >= 3 && anchor == TGL_ANCHOR_ROOT ? ws.t0[(h - 1) & 1] : nullptr;
            a.p_groups_static = h == 2 ? num_roots * S : 0;
            a.p_groups_dyn = h == 2 ? nullptr : counts + (h - 2);
        }
        const bool multi = h == 1 && S > 1;
        const int G = pick_group(static_cast<int64_t>(a.windows) * k);
        const int64_t work = h == 1 ? num_roots : cap[h - 1];
        {
            ScopedTimer tm(h == 1 ? TGL_TIMER_HOP1 : TGL_TIMER_HOPN, st);
            launch_hop(G, mode, h == 1, multi, last, win, a, work, st);
        }
        if (launch_status() != TGL_OK) return TGL_EDEVICE;
        if (last) break;

        // ---- exclusive scan of this hop's group counts -> next hop's indices ----
        const int64_t groups_cap = h == 1 ? num_roots * S : cap[h - 1];
        const int64_t *groups_dyn = h == 1 ? nullptr : counts + (h - 1);
        const int64_t tiles = scan_tiles(groups_cap) > 0 ? scan_tiles(groups_cap) : 1;
        ScopedTimer tm(TGL_TIMER_COMPACT, st);
        group_scan_kernel<<<static_cast<unsigned>(tiles), kBlock, 0, st>>>(ws.cnt[h & 1], groups_cap, groups_dyn,
                                                                          ws.tile_off);
        launch_scan_partials(ws.tile_off, tiles, counts + h, st);
        if (launch_status() != TGL_OK) return TGL_EDEVICE;
    }
    return TGL_OK;
}

tgl_status tgl_pointers_reset(const tgl_tcsr *g, int32_t num_snapshots, uint32_t *pointers, void *stream) {
    if (!g || !pointers || num_snapshots < 1 || num_snapshots > TGL_MAX_SNAPSHOTS) return TGL_EINVAL;
    if (g->num_nodes < 1 || g->num_nodes > INT32_MAX || !g->indptr) return TGL_EINVAL;
    if (g->num_entries < 0 || g->num_entries > static_cast<int64_t>(UINT32_MAX)) return TGL_EINVAL;
    if ((reinterpret_cast<uintptr_t>(pointers) & 3u) != 0) return TGL_EINVAL;
    hipStream_t st = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();
    const int64_t n = (static_cast<int64_t>(num_snapshots) + 1) * g->num_nodes;
    int64_t blocks = (n + kBlock - 1) / kBlock;
    if (blocks > kMaxGrid) blocks = kMaxGrid;
    pointers_reset_kernel<<<static_cast<unsigned>(blocks), kBlock, 0, st>>>(g->indptr, g->num_nodes, g->num_entries,
                                                                          n, pointers);
    return launch_status();
}

tgl_status tgl_sample(const tgl_tcsr *g, const int32_t *roots, const float *root_ts,
                      int64_t num_roots, int32_t hops, const int32_t *fanouts, int32_t mode,
                      int32_t num_snapshots, float snapshot_len, uint64_t seed,
                      uint64_t root_base, const tgl_hop_out *outs, int64_t *counts,
                      void *workspace, size_t workspace_bytes, void *stream) {
    return tgl_sample_ex(g, roots, root_ts, num_roots, hops, fanouts, mode, num_snapshots, snapshot_len, seed,
                         root_base, nullptr, outs, counts, workspace, workspace_bytes, stream);
}

tgl_status tgl_sample_noalloc(const tgl_tcsr *g, const int32_t *roots, const float *root_ts,
                              int64_t num_roots, int32_t hops, const int32_t *fanouts, int32_t mode,
                              int32_t num_snapshots, float snapshot_len, uint64_t seed,
                              uint64_t root_base, const tgl_hop_out *outs, int64_t *counts, void *stream) {
    int64_t cap[TGL_MAX_HOPS + 1];
    const tgl_status chk = sample_check(g, roots, root_ts, num_roots, hops, fanouts, mode, num_snapshots,
                                        snapshot_len, nullptr, outs, counts, cap);
    if (chk != TGL_OK) return chk;
    if (carve_sample_ws(nullptr, hops, cap, num_snapshots).bytes > TGL_NOALLOC_SCRATCH_BYTES) return TGL_ENOSPACE;
    void *ws = nullptr;
    if (scratch_ptr(&ws) != TGL_OK) return TGL_EDEVICE;
    return tgl_sample_ex(g, roots, root_ts, num_roots, hops, fanouts, mode, num_snapshots, snapshot_len, seed,
                         root_base, nullptr, outs, counts, ws, TGL_NOALLOC_SCRATCH_BYTES, stream);
}

}  // extern "C"
