/*
 * tgl_oracle.c -- plain, slow, single-threaded CPU oracle for the temporal
 * neighbour sampler over a Temporal-CSR (T-CSR).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; it exists so that tests, the smoke check and the CPU
 * baseline leg of the benchmark can state what the GPU library must return.
 * It shares no code, header or constant table with the GPU library.
 *
 * What it computes (paper: "TGL: A General Framework for Temporal GNN
 * Training on Billion-Scale Graphs", Zhou et al., VLDB 2022):
 *
 *  oracle_build  -- the T-CSR of Section 3.1 ("The T-CSR Data Structure"):
 *                   an indptr array of |V|+1 offsets and, per node, its
 *                   outgoing edges (neighbour, edge id, timestamp) sorted by
 *                   timestamp.  Ties in timestamp keep input order.  Plain
 *                   stable counting sort by node, then a stable merge sort of
 *                   each run by timestamp.
 *  oracle_locate -- the candidate window of a root inside one snapshot:
 *                   the edges of node x with  t - (s+1)*D <= ts < t - s*D
 *                   (Section 3 on dynamic snapshots built from the target
 *                   node's time; Section 3.1 "Sampling" and the strictness
 *                   rule that sampled neighbours are older than the root).
 *  oracle_sample -- Algorithm 1 (Parallel Temporal Sampler), run serially:
 *                   for each layer and snapshot, locate the window, draw
 *                   k_l neighbours (most recent, or uniform with
 *                   replacement), and feed the sampled neighbours with their
 *                   edge timestamps to the next layer (Section 3.1, the
 *                   multi-hop note on TGAT-style sampling).
 *
 * Readings of points the paper leaves open (documented in the design notes):
 *  - window s = 0 is the newest snapshot [t - D, t); with no snapshots the
 *    single window is (-inf, t)  (D = +inf, one snapshot);
 *  - window bounds are evaluated in IEEE double: hi = t - s*D (hi = t when
 *    s == 0), lo = t - (s+1)*D (lo = -inf when D is infinite); an entry is a
 *    candidate iff lo <= ts < hi, compared in double;
 *  - most recent: slot j takes the j-th newest candidate, PAD when fewer;
 *  - uniform: each slot draws independently (with replacement) the
 *    candidate  lo + floor(H * n / 2^64)  where H is the SplitMix64-finalizer
 *    hash of (seed, path, hop, window, slot); all slots PAD when n == 0;
 *  - dt = t - ts rounded to float32 (computed in double, then rounded once:
 *    with 53 >= 2*24 + 2 bits this equals the float32 subtraction);
 *  - PAD slot = (nbr -1, eid -1, ts -1.0f, dt -1.0f);
 *  - next-layer roots are the valid slots in output order; a root of layer
 *    h >= 2 samples only the window it inherited, relative to its own time;
 *  - path of a layer-1 root r is root_base + r; a child of layer-1 slot
 *    (r, s, j) has path  path*S*k1 + s*k1 + j;  a child of layer-h slot
 *    (q, j), h >= 2, has path  path*k_h + j  (all mod 2^64).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK      0
#define ORACLE_EINVAL -1
#define ORACLE_ERANGE -2
#define ORACLE_ENOMEM -5

#define ORACLE_MOST_RECENT 0
#define ORACLE_UNIFORM     1

/* ------------------------------------------------------------------------ */
/* T-CSR build (Section 3.1, "The T-CSR Data Structure")                    */
/* ------------------------------------------------------------------------ */

/* One directed entry of the T-CSR before ordering. */
typedef struct {
    int32_t v;      /* neighbour                                 */
    float   t;      /* timestamp                                 */
    int64_t e;      /* caller's edge id                          */
} oracle_entry;

/* Stable merge sort of ent[0..n) by timestamp (tmp has room for n).  Equal
 * timestamps keep their relative order.  Halves that are already in order
 * are not merged again. */
static void merge_sort_by_time(oracle_entry *ent, oracle_entry *tmp, int64_t n)
{
    for (int64_t width = 1; width < n; width *= 2) {
        for (int64_t lo = 0; lo + width < n; lo += 2 * width) {
            int64_t mid = lo + width;
            int64_t hi = lo + 2 * width < n ? lo + 2 * width : n;
            if (!(ent[mid].t < ent[mid - 1].t)) continue;     /* already in order */
            int64_t i = lo, j = mid, k = 0;
            while (i < mid && j < hi) {
                if (ent[j].t < ent[i].t) tmp[k++] = ent[j++];  /* ties: left first */
                else tmp[k++] = ent[i++];
            }
            while (i < mid) tmp[k++] = ent[i++];
            while (j < hi) tmp[k++] = ent[j++];
            memcpy(ent + lo, tmp, (size_t)k * sizeof(oracle_entry));
        }
    }
}

/* Entries: the m0 given edges (owner src, neighbour dst), then, when
 * undirected, the same edges reversed (owner dst, neighbour src) at positions
 * m0..2*m0-1.  The T-CSR orders them by owner node, then timestamp, then
 * position: a stable counting sort by owner (so each run keeps position
 * order) followed by a stable sort of every run by timestamp.  Returns the
 * number of entries written, or a negative status. */
int64_t oracle_build(int64_t m0, const int32_t *src, const int32_t *dst,
                     const float *ts, const int64_t *eid, int64_t num_nodes,
                     int undirected, int64_t *indptr, int32_t *nbr,
                     int64_t *eid_out, float *ts_out)
{
    if (m0 < 0 || num_nodes < 1 || num_nodes > INT32_MAX) return ORACLE_EINVAL;
    if (m0 > 0 && (!src || !dst || !ts)) return ORACLE_EINVAL;
    int64_t m = undirected ? 2 * m0 : m0;

    for (int64_t i = 0; i < m0; i++) {
        if (src[i] < 0 || src[i] >= num_nodes) return ORACLE_ERANGE;
        if (dst[i] < 0 || dst[i] >= num_nodes) return ORACLE_ERANGE;
        if (isnan(ts[i])) return ORACLE_ERANGE;
    }

    /* indptr[x] = number of entries whose owner is < x */
    memset(indptr, 0, (size_t)(num_nodes + 1) * sizeof(int64_t));
    for (int64_t i = 0; i < m; i++) {
        int32_t u = i < m0 ? src[i] : dst[i - m0];
        indptr[u + 1] += 1;
    }
    for (int64_t x = 0; x < num_nodes; x++) indptr[x + 1] += indptr[x];

    oracle_entry *ent = (oracle_entry *)malloc((size_t)(m > 0 ? m : 1) * sizeof(oracle_entry));
    oracle_entry *tmp = (oracle_entry *)malloc((size_t)(m > 0 ? m : 1) * sizeof(oracle_entry));
    int64_t *fill = (int64_t *)malloc((size_t)num_nodes * sizeof(int64_t));
    if (!ent || !tmp || !fill) { free(ent); free(tmp); free(fill); return ORACLE_ENOMEM; }
    memcpy(fill, indptr, (size_t)num_nodes * sizeof(int64_t));
    for (int64_t i = 0; i < m; i++) {           /* in position order */
        int64_t k = i < m0 ? i : i - m0;
        int fwd = i < m0;
        int32_t u = fwd ? src[k] : dst[k];
        oracle_entry en;
        en.v = fwd ? dst[k] : src[k];
        en.t = ts[k] == 0.0f ? 0.0f : ts[k];   /* -0 is stored as +0 */
        en.e = eid ? eid[k] : k;
        ent[fill[u]++] = en;
    }
    for (int64_t x = 0; x < num_nodes; x++)
        merge_sort_by_time(ent + indptr[x], tmp, indptr[x + 1] - indptr[x]);

    for (int64_t p = 0; p < m; p++) {
        nbr[p] = ent[p].v;
        eid_out[p] = ent[p].e;
        ts_out[p] = ent[p].t;
    }
    free(ent);
    free(tmp);
    free(fill);
    return m;
}

/* ------------------------------------------------------------------------ */
/* Window location (Section 3 dynamic snapshots; Section 3.1 "Sampling")   */
/* ------------------------------------------------------------------------ */

/* Number of positions p in [a, b) with ts[p] < v, for a run sorted
 * ascending.  Binary search; a NaN bound makes every comparison false and
 * gives a. */
static int64_t first_not_below(const float *ts, int64_t a, int64_t b, double v)
{
    int64_t lo = a, hi = b;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if ((double)ts[mid] < v) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

static double window_hi(float t, int32_t s, float delta)
{
    if (s == 0) return (double)t;
    return (double)t - (double)s * (double)delta;
}

static double window_lo(float t, int32_t s, float delta)
{
    if (isinf(delta)) return -INFINITY;
    return (double)t - (double)(s + 1) * (double)delta;
}

/* Candidate window [*lo, *hi) of node x between the bounds v_lo <= ts < v_hi.
 * A node outside [0, num_nodes) has an empty window at position 0. */
static void locate_bounds(int64_t num_nodes, const int64_t *indptr, const float *ts,
                          int32_t x, double v_lo, double v_hi, int64_t *lo, int64_t *hi)
{
    if (x < 0 || x >= num_nodes) { *lo = 0; *hi = 0; return; }
    int64_t a = indptr[x], b = indptr[x + 1];
    int64_t h = first_not_below(ts, a, b, v_hi);
    int64_t l = first_not_below(ts, a, b, v_lo);
    if (l > h) l = h;            /* keeps n = hi - lo >= 0 for any bound pair */
    *lo = l;
    *hi = h;
}

/* Candidate window [*lo, *hi) of root (x, t) in snapshot s. */
void oracle_locate(int64_t num_nodes, const int64_t *indptr, const float *ts,
                   int32_t x, float t, int32_t s, float delta,
                   int64_t *lo, int64_t *hi)
{
    locate_bounds(num_nodes, indptr, ts, x, window_lo(t, s, delta), window_hi(t, s, delta), lo, hi);
}

/* Batch form for tests: windows of n roots in snapshots s[i]. */
void oracle_locate_many(int64_t num_nodes, const int64_t *indptr, const float *ts,
                        int64_t n, const int32_t *x, const float *t,
                        const int32_t *s, float delta, int64_t *lo, int64_t *hi)
{
    for (int64_t i = 0; i < n; i++)
        oracle_locate(num_nodes, indptr, ts, x[i], t[i], s[i], delta, &lo[i], &hi[i]);
}

/* ------------------------------------------------------------------------ */
/* Counter-based draws: SplitMix64 finalizer (Steele, Lea, Flood, OOPSLA     */
/* 2014; the "mix64" variant with shifts 30/27/31).                          */
/* ------------------------------------------------------------------------ */

uint64_t oracle_mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t oracle_slot_hash(uint64_t seed, uint64_t path, int32_t hop, int32_t s, int32_t j)
{
    uint64_t key = ((uint64_t)(uint32_t)hop << 40) | ((uint64_t)(uint32_t)s << 24) | (uint64_t)(uint32_t)j;
    return oracle_mix64(oracle_mix64(oracle_mix64(seed ^ 0x9E3779B97F4A7C15ULL) ^ path) ^ key);
}

/* floor(h * n / 2^64): an index in [0, n) */
static int64_t scale_draw(uint64_t h, int64_t n)
{
    return (int64_t)(((unsigned __int128)h * (unsigned __int128)(uint64_t)n) >> 64);
}

/* ------------------------------------------------------------------------ */
/* Algorithm 1, serial                                                      */
/* ------------------------------------------------------------------------ */

/*
 * Inputs: T-CSR (indptr[num_nodes+1], nbr/eid/ts[entries]); R roots with
 * query times; hops L (1..8) with fanouts k[0..L-1]; mode; S snapshots of
 * length delta (S = 1 and delta = +inf: no snapshots); seed; root_base.
 *
 * Outputs, for hop h = 1..L (index h-1), caller-allocated with capacity
 *   slots_h = R*S*k1*k2*...*k_h:
 *   o_nbr[h-1], o_eid[h-1], o_ts[h-1], o_dt[h-1]  -- slot arrays
 *   o_parent[h-1]   -- for h >= 2: index of the hop-(h-1) slot each root of
 *                      hop h came from (ignored for h = 1, may be NULL)
 *   counts[h-1]     -- number of roots of hop h (counts[0] = R)
 * Hop 1 slot (r, s, j) is at (r*S + s)*k1 + j; hop h >= 2 slot (q, j) at
 * q*k_h + j.
 */
/*
 * anchor selects the snapshot windows of a root of hop h >= 2 (the paper
 * creates snapshots from the target nodes' timestamps, Section 3, and
 * searches them at later layers, Algorithm 1):
 *   0 -- relative to the root's own time t (its parent slot's timestamp):
 *        [t - (s+1)D, t - sD);
 *   1 -- relative to the time t0 of the hop-1 root it descends from, and
 *        before its own time: [t0 - (s+1)D, min(t0 - sD, t)).
 * Hop 1 is the same under both (t0 = t).
 */
int oracle_sample_anchored(int64_t num_nodes, const int64_t *indptr, const int32_t *nbr,
                           const int64_t *eid, const float *ts,
                           int64_t num_roots, const int32_t *roots, const float *root_ts,
                           int32_t hops, const int32_t *fanouts, int32_t mode,
                           int32_t num_snapshots, float delta, uint64_t seed,
                           uint64_t root_base, int32_t anchor,
                           int32_t *const *o_nbr, int64_t *const *o_eid,
                           float *const *o_ts, float *const *o_dt,
                           int64_t *const *o_parent, int64_t *counts)
{
    if (anchor != 0 && anchor != 1) return ORACLE_EINVAL;
    if (num_nodes < 1 || num_roots < 0 || hops < 1 || hops > 8) return ORACLE_EINVAL;
    if (mode != ORACLE_MOST_RECENT && mode != ORACLE_UNIFORM) return ORACLE_EINVAL;
    if (num_snapshots < 1 || isnan(delta) || !(delta > 0.0f)) return ORACLE_EINVAL;
    if (isinf(delta) && num_snapshots != 1) return ORACLE_EINVAL;
    for (int h = 0; h < hops; h++)
        if (fanouts[h] < 1 || fanouts[h] > 1024) return ORACLE_EINVAL;

    const int32_t S = num_snapshots;

    /* roots of the current hop */
    int64_t n_cur = num_roots;
    int32_t *cx = (int32_t *)malloc((size_t)(n_cur > 0 ? n_cur : 1) * sizeof(int32_t));
    float *ct = (float *)malloc((size_t)(n_cur > 0 ? n_cur : 1) * sizeof(float));
    int32_t *cs = (int32_t *)malloc((size_t)(n_cur > 0 ? n_cur : 1) * sizeof(int32_t));
    uint64_t *cp = (uint64_t *)malloc((size_t)(n_cur > 0 ? n_cur : 1) * sizeof(uint64_t));
    float *ca = (float *)malloc((size_t)(n_cur > 0 ? n_cur : 1) * sizeof(float));   /* hop-1 ancestor time */
    if (!cx || !ct || !cs || !cp || !ca) return ORACLE_ENOMEM;
    for (int64_t r = 0; r < num_roots; r++) {
        cx[r] = roots[r];
        ct[r] = root_ts[r];
        cs[r] = 0;
        cp[r] = root_base + (uint64_t)r;
        ca[r] = root_ts[r];
    }

    for (int32_t h = 1; h <= hops; h++) {
        const int32_t k = fanouts[h - 1];
        const int32_t wins = (h == 1) ? S : 1;          /* windows per root */
        counts[h - 1] = n_cur;

        int64_t n_slots = n_cur * wins * k;
        int32_t *nx = NULL; float *nt = NULL; int32_t *ns = NULL; uint64_t *np_ = NULL; float *na = NULL;
        int64_t n_next = 0;
        if (h < hops) {
            size_t cap = (size_t)(n_slots > 0 ? n_slots : 1);
            nx = (int32_t *)malloc(cap * sizeof(int32_t));
            nt = (float *)malloc(cap * sizeof(float));
            ns = (int32_t *)malloc(cap * sizeof(int32_t));
            np_ = (uint64_t *)malloc(cap * sizeof(uint64_t));
            na = (float *)malloc(cap * sizeof(float));
            if (!nx || !nt || !ns || !np_ || !na) return ORACLE_ENOMEM;
        }

        for (int64_t q = 0; q < n_cur; q++) {
            for (int32_t w = 0; w < wins; w++) {
                int32_t s = (h == 1) ? w : cs[q];
                int64_t lo, hi;
                if (h >= 2 && anchor == 1) {
                    double v_hi = window_hi(ca[q], s, delta);
                    if ((double)ct[q] < v_hi) v_hi = (double)ct[q];
                    locate_bounds(num_nodes, indptr, ts, cx[q], window_lo(ca[q], s, delta), v_hi, &lo, &hi);
                } else {
                    oracle_locate(num_nodes, indptr, ts, cx[q], ct[q], s, delta, &lo, &hi);
                }
                int64_t n = hi - lo;
                for (int32_t j = 0; j < k; j++) {
                    int64_t slot = (q * wins + w) * (int64_t)k + j;
                    int64_t p = -1;
                    if (mode == ORACLE_MOST_RECENT) {
                        if (j < n) p = hi - 1 - j;
                    } else {
                        if (n > 0) p = lo + scale_draw(oracle_slot_hash(seed, cp[q], h, s, j), n);
                    }
                    if (p < 0) {
                        o_nbr[h - 1][slot] = -1;
                        o_eid[h - 1][slot] = -1;
                        o_ts[h - 1][slot] = -1.0f;
                        o_dt[h - 1][slot] = -1.0f;
                        continue;
                    }
                    o_nbr[h - 1][slot] = nbr[p];
                    o_eid[h - 1][slot] = eid[p];
                    o_ts[h - 1][slot] = ts[p];
                    o_dt[h - 1][slot] = (float)((double)ct[q] - (double)ts[p]);
                    if (h < hops) {
                        nx[n_next] = nbr[p];
                        nt[n_next] = ts[p];
                        ns[n_next] = s;
                        na[n_next] = ca[q];
                        np_[n_next] = (h == 1)
                            ? cp[q] * (uint64_t)S * (uint64_t)k + (uint64_t)s * (uint64_t)k + (uint64_t)j
                            : cp[q] * (uint64_t)k + (uint64_t)j;
                        o_parent[h][n_next] = slot;
                        n_next++;
                    }
                }
            }
        }

        free(cx); free(ct); free(cs); free(cp); free(ca);
        if (h == hops) { cx = NULL; break; }
        cx = nx; ct = nt; cs = ns; cp = np_; ca = na;
        n_cur = n_next;
    }
    return ORACLE_OK;
}

/* Algorithm 1 with every window relative to its root's own time. */
int oracle_sample(int64_t num_nodes, const int64_t *indptr, const int32_t *nbr,
                  const int64_t *eid, const float *ts,
                  int64_t num_roots, const int32_t *roots, const float *root_ts,
                  int32_t hops, const int32_t *fanouts, int32_t mode,
                  int32_t num_snapshots, float delta, uint64_t seed,
                  uint64_t root_base,
                  int32_t *const *o_nbr, int64_t *const *o_eid,
                  float *const *o_ts, float *const *o_dt,
                  int64_t *const *o_parent, int64_t *counts)
{
    return oracle_sample_anchored(num_nodes, indptr, nbr, eid, ts, num_roots, roots, root_ts, hops,
                                  fanouts, mode, num_snapshots, delta, seed, root_base, 0,
                                  o_nbr, o_eid, o_ts, o_dt, o_parent, counts);
}

int oracle_version(void) { return 1; }
