/*
 * tgl.h -- C ABI of libtgl: a Temporal-CSR (T-CSR) build and a multi-hop
 * temporal neighbour sampler on one AMD Instinct MI355X (gfx950) GPU.
 *
 * Method: "TGL: A General Framework for Temporal GNN Training on
 * Billion-Scale Graphs" (Zhou et al., VLDB 2022), Section 3.1 (the T-CSR data
 * structure, sampling, parallel sampling) and Algorithm 1 (Parallel Temporal
 * Sampler), with dynamic snapshots as described at the start of Section 3.
 *
 * Conventions for every entry point:
 *  - Array arguments marked [device] are device pointers on the current HIP
 *    device; [host] pointers are ordinary host memory read during the call.
 *  - The caller owns every buffer (inputs, T-CSR arrays, outputs and
 *    workspace).  The library allocates no device memory in these calls.
 *  - Work is enqueued on `stream` (a hipStream_t passed as void*; NULL means
 *    the null stream).  Device inputs must stay valid, and outputs must not be
 *    read, until that work completes.
 *  - Functions return a tgl_status and never throw.  Argument checks run on
 *    the host before anything is enqueued; a failed check enqueues nothing.
 *  - Calls that overlap on one stream are ordered; calls on different
 *    streams must not share outputs or workspace.
 */
#ifndef TGL_H
#define TGL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t tgl_status;
#define TGL_OK        0   /* success                                           */
#define TGL_EINVAL   (-1) /* invalid argument (checked on the host)            */
#define TGL_ERANGE   (-2) /* build input out of range: endpoint not in [0,N) or
                             NaN timestamp (found on the device)                */
#define TGL_ENOSPACE (-3) /* workspace smaller than the matching *_workspace() */
#define TGL_EDEVICE  (-4) /* a HIP call or kernel launch failed                */

#define TGL_MOST_RECENT 0 /* k newest candidates, newest first (Sec. 2.3)     */
#define TGL_UNIFORM     1 /* k independent uniform draws from the candidates   */

#define TGL_BUILD_UNDIRECTED 1u /* also insert every edge reversed             */

#define TGL_MAX_HOPS      8
#define TGL_MAX_FANOUT    1024
#define TGL_MAX_SNAPSHOTS 64
#define TGL_INDEX_STRIDE  32   /* entries per sample of the search index */

/*
 * One T-CSR entry: an edge leaving the owner node (whose run contains the
 * entry) towards node `nbr & TGL_NBR_MASK`, at time `ts`, with the caller's
 * edge id `eid`.  Section 3.1 keeps indices and times as separate arrays;
 * here they are interleaved into one 16-byte record so that a sampled slot is
 * fetched with a single aligned 16-byte load.
 *
 * Node ids are below 2^31, so bit 31 of `nbr` is free; it holds a hint,
 * TGL_NBR_FIRST: when set, the neighbour's own run has no entry with a
 * timestamp below this entry's ts.  A later hop's root (nbr, ts) then has an
 * empty window whatever its snapshot, because every window lies below the
 * root's time, so the sampler skips the neighbour's node record.  A clear bit
 * promises nothing: results are the same with the bit set exactly as defined
 * or clear everywhere.  tgl_tcsr_build sets it exactly; tgl_tcsr_nodes can
 * set it for a T-CSR built elsewhere.
 */
#define TGL_NBR_MASK  0x7fffffffu
#define TGL_NBR_FIRST 0x80000000u
typedef struct tgl_entry {
    int32_t nbr;
    float ts;
    int64_t eid;
} tgl_entry;

/*
 * Summary of one node's run, one 128-byte record (one cache line) per node:
 * the run occupies entries [start, end); first_ts and last_ts are the
 * timestamps of its first and last entry (+inf and -inf for an empty run);
 * ts[i] is the timestamp of entry start + i for i < min(end - start,
 * TGL_NODE_INLINE), +inf beyond.  The sampler reads it in place of the indptr
 * pair.  A window edge at or below first_ts, or above last_ts, is then
 * resolved without reading the run -- the O(1) candidate location that
 * Section 3.1 obtains from per-node pointer arrays, kept here as stateless
 * per-node data -- and a run of at most TGL_NODE_INLINE entries is searched
 * inside the same line.
 */
#define TGL_NODE_INLINE 28
typedef struct tgl_node {
    uint32_t start;
    uint32_t end;
    float first_ts;
    float last_ts;
    float ts[TGL_NODE_INLINE];
} tgl_node;

/*
 * The neighbour's history before an entry: for entry p = (owner u, neighbour
 * v, time t), the positions [lo, hi) of v's own run whose timestamps are
 * below t, i.e. lo = indptr[v] and hi = lo + #{entries of v with ts < t}
 * ({0, 0} for a neighbour id outside [0, num_nodes)).  A root of a later hop
 * made from this entry is (v, t), and without snapshots its candidates are
 * exactly these entries: the search Algorithm 1 runs for layers > 0, done
 * once per entry when the T-CSR is built.  With it, the sampler gathers an
 * entry's span together with the entry and serves the next hop's root
 * without reading its node record or searching its run.  hi == lo is the
 * TGL_NBR_FIRST hint.
 */
typedef struct tgl_span {
    uint32_t lo;
    uint32_t hi;
} tgl_span;

/*
 * One cell of a run's time directory.  Section 3.1 finds a window edge by a
 * binary search of the node's time-sorted run; the directory replaces most
 * of that search by one lookup.  The run [a, b) of a node (first and last
 * timestamps f, l) owns the search-index slots j with j * TGL_INDEX_STRIDE
 * in [a, b): K = ceil(b / S) - ceil(a / S) of them (S = TGL_INDEX_STRIDE),
 * and slot ceil(a / S) + k holds its cell k.  The cells split [f, l] evenly:
 * with sc = K / (l - f) when l - f is positive and finite (sc = 0 otherwise),
 *   cell(t) = 0 if t <= f;  K - 1 if t >= l;
 *             min(K - 1, floor((t - f) * sc)) otherwise,
 * every operation a float32 one rounded to nearest.  cell is non-decreasing
 * in t, so each cell's entries are one stretch of the run, and cell k holds
 *   pos = a + #{entries of the run whose timestamp's cell is below k}
 *   ts  = the timestamp of entry pos (+inf if pos = b).
 * For a threshold v with cell(v) = k, the count of the run's timestamps
 * below v lies between pos and the next cell's pos (b after the last cell),
 * and equals pos when v <= ts.
 */
typedef struct tgl_cell {
    uint32_t pos;
    float ts;
} tgl_cell;

/*
 * Non-owning view of a T-CSR (Section 3.1): node x owns entries
 * [indptr[x], indptr[x+1]) of `entries`, sorted by ts ascending (ties in any
 * fixed order; tgl_tcsr_build uses input order).  Timestamps must not be NaN.
 *   indptr   [device] int64[num_nodes + 1], indptr[0] = 0, non-decreasing,
 *                     indptr[num_nodes] = num_entries
 *   entries  [device] tgl_entry[num_entries], 16-byte aligned
 *   ts       [device] float[num_entries], 16-byte aligned: ts[p] equals
 *                     entries[p].ts.  The window search reads only this array
 *                     (4 bytes per entry), the gather only `entries`.
 *   nodes    [device] tgl_node[num_nodes], 128-byte aligned: the summary of
 *                     each run (start = indptr[x], end = indptr[x+1]); see
 *                     tgl_tcsr_nodes for a T-CSR built elsewhere.
 *   ts_index [device] float[tgl_index_len(num_entries)], 16-byte aligned, or
 *                     NULL: ts_index[j] = ts[j * TGL_INDEX_STRIDE].  A search
 *                     over a long run first narrows on this array (1/32 of the
 *                     timestamps, small enough to stay in cache), then reads
 *                     at most TGL_INDEX_STRIDE - 1 timestamps of the run.
 *                     Results are the same with or without it.
 *   hist     [device] tgl_span[num_entries], 8-byte aligned, or NULL: the
 *                     neighbour's history before each entry (see tgl_span).
 *                     Read by calls with one snapshot of infinite length and
 *                     more than one hop; results are the same with or
 *                     without it.
 *   dir      [device] tgl_cell[tgl_index_len(num_entries)], 8-byte aligned,
 *                     or NULL: the time directory of every run (see
 *                     tgl_cell), written by tgl_tcsr_build or tgl_tcsr_nodes
 *                     from the same arrays.  The window search of a run
 *                     longer than a few cache lines starts from it; results
 *                     are the same with or without it.
 * num_entries must be at most 2^32 - 1.  The sampler clamps every indptr
 * value into [0, num_entries], so a malformed view yields wrong samples but
 * never an out-of-bounds access.
 */
typedef struct tgl_tcsr {
    int64_t num_nodes;
    int64_t num_entries;
    const int64_t *indptr;
    const tgl_entry *entries;
    const float *ts;
    const tgl_node *nodes;
    const float *ts_index;
    const tgl_span *hist;
    const tgl_cell *dir;
} tgl_tcsr;

/*
 * Outputs of one hop (structure of arrays, one element per slot).
 *   nbr, eid, ts, dt  [device] slot arrays with capacity
 *                     tgl_sample_capacity(..., hop) elements each
 *   parent            [device] int64, one per root of this hop: index of the
 *                     previous hop's slot the root came from.  Capacity
 *                     tgl_sample_capacity(..., hop - 1).  Unused (may be NULL)
 *                     for hop 1.
 * A missing neighbour (PAD) is nbr = -1, eid = -1, ts = -1.0f, dt = -1.0f.
 */
typedef struct tgl_hop_out {
    int32_t *nbr;
    int64_t *eid;
    float *ts;
    float *dt;
    int64_t *parent;
} tgl_hop_out;

/* Library version (major * 10000 + minor * 100 + patch). */
int32_t tgl_version(void);

/* Static string naming a status code. */
const char *tgl_status_str(tgl_status status);

/* ------------------------------------------------------------------------ */
/* T-CSR build (Section 3.1, "The T-CSR Data Structure"; Figure 3)          */
/* ------------------------------------------------------------------------ */

/*
 * Bytes of workspace tgl_tcsr_build needs for `num_edges` input edges on
 * `num_nodes` nodes with `flags`.  Returns 0 for arguments tgl_tcsr_build
 * would reject with TGL_EINVAL.
 */
size_t tgl_tcsr_build_workspace(int64_t num_edges, int64_t num_nodes, uint32_t flags);

/*
 * Builds the T-CSR of a temporal edge list.
 *   src, dst   [device] int32[num_edges]   endpoints, each in [0, num_nodes)
 *   ts         [device] float[num_edges]   timestamps, not NaN (-0 is stored
 *                                           as +0)
 *   eid        [device] int64[num_edges]   edge ids, or NULL for eid = index
 *   num_edges  >= 0; entries M = num_edges, or 2*num_edges with
 *              TGL_BUILD_UNDIRECTED; M must be < 2^32
 *   num_nodes  in [1, 2^31 - 1]
 *   flags      0 or TGL_BUILD_UNDIRECTED
 *   indptr     [device] int64[num_nodes + 1]  output
 *   entries    [device] tgl_entry[M]          output, 16-byte aligned
 *   ts_out     [device] float[M]              output, 16-byte aligned: the
 *                                             entries' timestamps again
 *   nodes_out  [device] tgl_node[num_nodes]   output, 128-byte aligned
 *   ts_index_out [device] float[tgl_index_len(M)] output, 16-byte aligned, or
 *                                             NULL (no search index)
 *   hist_out   [device] tgl_span[M]           output, 8-byte aligned, or NULL
 *                                             (no neighbour histories)
 *   dir_out    [device] tgl_cell[tgl_index_len(M)] output, 8-byte aligned,
 *                                             or NULL (no time directory)
 *   workspace  [device] at least tgl_tcsr_build_workspace(...) bytes
 * Entry i < num_edges is (owner src[i], nbr dst[i], ts[i], eid[i]); with
 * TGL_BUILD_UNDIRECTED entry num_edges + i is the reversed edge (owner
 * dst[i], nbr src[i]).  Each node's run is sorted by (ts, entry index).
 * Every entry's TGL_NBR_FIRST bit is set exactly as defined at tgl_entry.
 * Synchronises `stream` once, to read the device-side range check; returns
 * TGL_ERANGE (outputs unspecified) if any endpoint or timestamp is invalid.
 */
tgl_status tgl_tcsr_build(const int32_t *src, const int32_t *dst, const float *ts,
                          const int64_t *eid, int64_t num_edges, int64_t num_nodes,
                          uint32_t flags, int64_t *indptr, tgl_entry *entries, float *ts_out,
                          tgl_node *nodes_out, float *ts_index_out, tgl_span *hist_out,
                          tgl_cell *dir_out, void *workspace, size_t workspace_bytes, void *stream);

/* Length of the search index of a T-CSR with num_entries entries:
 * ceil(num_entries / TGL_INDEX_STRIDE), or -1 if num_entries is negative. */
int64_t tgl_index_len(int64_t num_entries);

/*
 * Writes the per-node summaries, the search index (if ts_index is not NULL),
 * the TGL_NBR_FIRST hints (if entries is not NULL), the neighbour histories
 * (if hist is not NULL) and the time directory (if dir is not NULL) of a
 * T-CSR given by its indptr, timestamp and entry arrays (for a T-CSR built
 * elsewhere and uploaded).
 *   indptr     [device] int64[num_nodes + 1]
 *   ts         [device] float[num_entries]
 *   num_nodes  in [1, 2^31 - 1];  num_entries in [0, 2^32 - 1]
 *   nodes      [device] tgl_node[num_nodes], 128-byte aligned, output
 *   ts_index   [device] float[tgl_index_len(num_entries)], 16-byte aligned,
 *              output, or NULL
 *   entries    [device] tgl_entry[num_entries], 16-byte aligned, or NULL:
 *              bit 31 of each nbr is rewritten (set exactly when the
 *              neighbour's run has no timestamp below the entry's ts; clear
 *              for a neighbour id outside [0, num_nodes)), the other fields
 *              are left alone
 *   hist       [device] tgl_span[num_entries], 8-byte aligned, output, or
 *              NULL; requires entries
 *   dir        [device] tgl_cell[tgl_index_len(num_entries)], 8-byte
 *              aligned, output, or NULL
 * indptr values are clamped into [0, num_entries].  Never synchronises.
 */
tgl_status tgl_tcsr_nodes(const int64_t *indptr, const float *ts, int64_t num_nodes,
                          int64_t num_entries, tgl_node *nodes, float *ts_index,
                          tgl_entry *entries, tgl_span *hist, tgl_cell *dir, void *stream);

/*
 * Conversions between the entries and the column layout of Section 3.1's
 * T-CSR (separate neighbour, timestamp and edge-id arrays beside indptr), for
 * T-CSRs that arrive or leave in columns.
 *
 * tgl_tcsr_pack writes entries[p] = {nbr[p] with bit 31 clear, ts[p],
 * eid[p]} (eid NULL: p).  The hints stay clear; tgl_tcsr_nodes sets them
 * and writes the per-node data of the packed T-CSR.
 *   nbr, ts, eid  [device] int32 / float / int64 [num_entries]
 *   entries       [device] tgl_entry[num_entries], 16-byte aligned, output
 * tgl_tcsr_unpack writes the neighbour ids (bit 31 cleared) and edge ids of
 * the entries to nbr and eid, either of which may be NULL (the timestamps are
 * the T-CSR's ts array already).
 * num_entries in [0, 2^32 - 1].  Neither synchronises.
 */
tgl_status tgl_tcsr_pack(const int32_t *nbr, const float *ts, const int64_t *eid, int64_t num_entries,
                         tgl_entry *entries, void *stream);
tgl_status tgl_tcsr_unpack(const tgl_entry *entries, int64_t num_entries, int32_t *nbr, int64_t *eid,
                           void *stream);

/* ------------------------------------------------------------------------ */
/* Sampler (Algorithm 1; Section 3.1 "Sampling" and "Parallel Sampling")    */
/* ------------------------------------------------------------------------ */

/*
 * Worst-case number of slots of hop `hop` (1..hops): num_roots * S * k_1 *
 * ... * k_hop (S = num_snapshots).  hop = 0 gives num_roots.  Returns -1 for
 * invalid arguments or if the product exceeds 2^62.
 */
int64_t tgl_sample_capacity(int64_t num_roots, int32_t hops, const int32_t *fanouts,
                            int32_t num_snapshots, int32_t hop);

/* Bytes of workspace tgl_sample needs (0 for invalid arguments). */
size_t tgl_sample_workspace(int64_t num_roots, int32_t hops, const int32_t *fanouts,
                            int32_t num_snapshots);

/*
 * Samples `hops` layers of temporal neighbours for `num_roots` roots.
 *   g             [host] T-CSR view (arrays on the device)
 *   roots         [device] int32[num_roots]  root nodes; a node outside
 *                                            [0, num_nodes) gets only PAD
 *   root_ts       [device] float[num_roots]  query times (NaN gets only PAD)
 *   hops          1..TGL_MAX_HOPS
 *   fanouts       [host] int32[hops], each 1..TGL_MAX_FANOUT
 *   mode          TGL_MOST_RECENT or TGL_UNIFORM
 *   num_snapshots S in 1..TGL_MAX_SNAPSHOTS
 *   snapshot_len  D > 0; +inf means one unbounded window (then S must be 1)
 *   seed          key of the uniform draws
 *   root_base     global index of roots[0]; a call over roots [0, n) equals
 *                 calls over sub-ranges with root_base advanced accordingly
 *   outs          [host] tgl_hop_out[hops]
 *   counts        [device] int64[hops]: counts[h-1] = number of roots of hop h
 *   workspace     [device] at least tgl_sample_workspace(...) bytes
 *
 * Window s (0 = newest) of a root (x, t) holds the entries of x with
 *   t - (s+1)*D <= ts < t - s*D,
 * both bounds evaluated in double precision (upper bound t when s = 0, lower
 * bound -inf when D is infinite).  Hop 1 samples every window of every root:
 * slot (r, s, j) is at index (r*S + s)*k_1 + j.  The valid slots of hop h, in
 * index order, become the roots of hop h+1 (node = slot nbr, time = slot ts)
 * and sample only the window they came from, relative to their own time:
 * slot (q, j) is at q*k_{h+1} + j.
 *   TGL_MOST_RECENT: slot j is the j-th newest candidate, PAD if fewer.
 *   TGL_UNIFORM:     slot j is candidate floor(H * n / 2^64) (n candidates,
 *                    oldest first), all PAD if n = 0, where
 *                    H = mix(mix(mix(seed ^ 0x9E3779B97F4A7C15) ^ path) ^
 *                            (hop << 40 | s << 24 | j)),
 *                    mix = the SplitMix64 finalizer, path = root_base + r
 *                    for hop-1 roots, path*S*k_1 + s*k_1 + j for a child of
 *                    hop-1 slot (r, s, j), path*k_h + j for a child of
 *                    hop-h slot (q, j), all modulo 2^64.
 *   dt = t - ts rounded to float.
 * Never synchronises the stream; per-hop root counts stay on the device.
 */
tgl_status tgl_sample(const tgl_tcsr *g, const int32_t *roots, const float *root_ts,
                      int64_t num_roots, int32_t hops, const int32_t *fanouts, int32_t mode,
                      int32_t num_snapshots, float snapshot_len, uint64_t seed,
                      uint64_t root_base, const tgl_hop_out *outs, int64_t *counts,
                      void *workspace, size_t workspace_bytes, void *stream);

/*
 * tgl_sample for callers that cannot allocate device memory (code under HIP
 * graph capture, serving loops, harnesses that forbid allocation): the
 * workspace is a fixed area of TGL_NOALLOC_SCRATCH_BYTES bytes that the
 * library's code object holds on each GPU it is loaded on, until the process
 * ends.  Arguments, outputs and errors as tgl_sample, without the workspace;
 * a call whose tgl_sample_workspace(...) exceeds the area returns
 * TGL_ENOSPACE and enqueues nothing.  The call allocates nothing (the first
 * call on a device looks up the area's device address).  Every call on one
 * GPU uses that GPU's one area: calls that overlap on one GPU (several
 * streams or threads) race and must be serialised by the caller.  Nothing in
 * the area needs clearing between calls.
 */
#define TGL_NOALLOC_SCRATCH_BYTES (128u << 20)
tgl_status tgl_sample_noalloc(const tgl_tcsr *g, const int32_t *roots, const float *root_ts,
                              int64_t num_roots, int32_t hops, const int32_t *fanouts, int32_t mode,
                              int32_t num_snapshots, float snapshot_len, uint64_t seed,
                              uint64_t root_base, const tgl_hop_out *outs, int64_t *counts, void *stream);

/* Options of tgl_sample_ex (zero-initialise; NULL means all defaults). */
#define TGL_ANCHOR_OWN  0  /* windows of a hop >= 2 root at its own time t:
                              [t - (s+1) D, t - s D) (the default)              */
#define TGL_ANCHOR_ROOT 1  /* at the time t0 of its hop-1 ancestor, cut below
                              its own time: [t0 - (s+1) D, min(t0 - s D, t))    */
typedef struct tgl_sample_opts {
    int32_t anchor;        /* TGL_ANCHOR_OWN or TGL_ANCHOR_ROOT                   */
    int32_t reserved;      /* 0                                                  */
    uint32_t *pointers;    /* [device] (S + 1) x num_nodes saved window edges, or
                              NULL: see tgl_pointers_reset                       */
} tgl_sample_opts;

/*
 * tgl_sample with options.  The snapshot anchor chooses where the windows of
 * the roots of hops >= 2 sit.  The paper creates snapshots from the target
 * nodes' timestamps (Section 3) and searches "the snapshot S_s" at later
 * layers (Algorithm 1); TGL_ANCHOR_OWN reads the target of a later layer as
 * that layer's root (its own time, the neighbour's edge time), and
 * TGL_ANCHOR_ROOT as the mini-batch's root, keeping strict ts < t below the
 * parent.  Hop 1 is the same under both, and so is every hop when S = 1 and
 * D = +inf.  Other arguments, errors and outputs as tgl_sample; opts may be
 * NULL; an unknown anchor is TGL_EINVAL.
 */
tgl_status tgl_sample_ex(const tgl_tcsr *g, const int32_t *roots, const float *root_ts,
                         int64_t num_roots, int32_t hops, const int32_t *fanouts, int32_t mode,
                         int32_t num_snapshots, float snapshot_len, uint64_t seed,
                         uint64_t root_base, const tgl_sample_opts *opts, const tgl_hop_out *outs,
                         int64_t *counts, void *workspace, size_t workspace_bytes, void *stream);

/*
 * Per-node pointer arrays of Section 3.1 / Algorithm 1 for hop 1: entry
 * i * num_nodes + x is a saved position in node x's run for window edge i
 * (edge i at t - i * D, i = 0..S), which the sampler advances as roots come
 * in chronologically instead of searching the run from scratch.  On the GPU
 * they are an acceleration structure with no effect on results: hop 1 of a
 * tgl_sample_ex call with opts->pointers reads a node's saved position for
 * each edge it must locate in a run longer than 61 entries (the shorter ones
 * are one load anyway), loads the timestamps around it, falls back to a
 * search of the rest of the run if the edge is not among them, and raises
 * the saved position to the edge found (atomic maximum, so duplicate roots
 * in a batch need no locks).  Roots in chronological order per node make the
 * first load the answer, as in the paper; any order gives the same samples.
 *   pointers   [device] uint32[(num_snapshots + 1) * num_nodes], caller-owned,
 *              kept across calls for one T-CSR and one num_snapshots
 * tgl_pointers_reset sets every saved position to the start of its run (the
 * start of an epoch).  Never synchronises.
 */
tgl_status tgl_pointers_reset(const tgl_tcsr *g, int32_t num_snapshots, uint32_t *pointers, void *stream);

/* ------------------------------------------------------------------------ */
/* Message-flow-graph blocks of a hop (Algorithm 1, "generate DGL MFGs")    */
/* ------------------------------------------------------------------------ */

/*
 * One hop's sampled slots as a bipartite block for message passing, in
 * compressed sparse column form (edges grouped by destination):
 *   destination nodes  the hop's groups, G of them: hop 1 has one group per
 *                      (root, window), in root-major order; a later hop one
 *                      per root;
 *   edges              the valid slots, E of them, in slot order (a group's
 *                      valid slots are a prefix of its k slots);
 *   source nodes       the G destination nodes first, then one node per edge
 *                      (the sampled neighbour at its edge time: temporal
 *                      nodes are not merged), so edge e runs from source
 *                      G + e to its group.
 * Outputs (device arrays, capacities from groups_cap and k):
 *   indptr   int64[groups_cap + 1]  edges of group g: [indptr[g], indptr[g+1])
 *   edge_dst int64[groups_cap * k]  group of each edge, or NULL
 *   edge_eid int64[groups_cap * k]  edge id
 *   edge_dt  float[groups_cap * k]  time difference (the slot's dt)
 *   src_nid  int32[groups_cap * (k + 1)]  node of each source node
 *   src_ts   float[groups_cap * (k + 1)]  time of each source node
 *   sizes    int64[2]               G and E, written on the device
 * Only the first G + 1, E and G + E entries are written.
 */
typedef struct tgl_mfg {
    int64_t *indptr;
    int64_t *edge_dst;
    int64_t *edge_eid;
    float *edge_dt;
    int32_t *src_nid;
    float *src_ts;
    int64_t *sizes;
} tgl_mfg;

/* Workspace bytes for tgl_mfg_export with at most groups_cap groups (0 for a
 * negative count). */
size_t tgl_mfg_workspace(int64_t groups_cap);

/*
 * Builds the block of one hop from tgl_sample's outputs.
 *   hop        [host] the hop's tgl_hop_out (nbr, eid, ts, dt; parent for hop >= 2)
 *   prev       [host] the previous hop's tgl_hop_out (hop >= 2), or NULL for hop 1
 *   roots, root_ts  [device] the call's roots (hop 1: destination nodes); both
 *              NULL is accepted for a call with no roots (they are read only
 *              for groups below count * windows)
 *   count      [device] int64: roots of this hop (counts[h] of tgl_sample)
 *   windows    S for hop 1, 1 for a later hop
 *   k          the hop's fanout, in [1, TGL_MAX_FANOUT]
 *   groups_cap upper bound of count * windows (the output capacities)
 * Never synchronises.  Errors: TGL_EINVAL, TGL_ENOSPACE (workspace),
 * TGL_EDEVICE.
 */
tgl_status tgl_mfg_export(const tgl_hop_out *hop, const tgl_hop_out *prev, const int32_t *roots,
                          const float *root_ts, const int64_t *count, int32_t windows, int32_t k,
                          int64_t groups_cap, const tgl_mfg *out, void *workspace, size_t workspace_bytes,
                          void *stream);

/* ------------------------------------------------------------------------ */
/* Feature / state gather for sampled slots (Figure 2, steps 2 and 3)       */
/* ------------------------------------------------------------------------ */

#define TGL_KEY_NODE   0   /* rows indexed by the slot's neighbour id (nbr)   */
#define TGL_KEY_EDGE   1   /* rows indexed by the slot's edge id (eid)        */
#define TGL_MAX_TABLES 8
#define TGL_MAX_ROW_BYTES 65536

/*
 * One table of fixed-size rows (node features, node memory, mailbox, edge
 * features, ...) and the output it is gathered into.
 *   rows       [device] num_rows x row_bytes, 16-byte aligned
 *   out        [device] n x row_bytes (n of tgl_gather), 16-byte aligned
 *   num_rows   >= 0
 *   row_bytes  multiple of 16 in [16, TGL_MAX_ROW_BYTES]; any element type
 *   key        TGL_KEY_NODE or TGL_KEY_EDGE
 */
typedef struct tgl_table {
    const void *rows;
    void *out;
    int64_t num_rows;
    int32_t row_bytes;
    int32_t key;
} tgl_table;

/*
 * For every slot i < n and every table T: T.out[i] = T.rows[key_i], where
 * key_i is nbr[i] (TGL_KEY_NODE) or eid[i] (TGL_KEY_EDGE); a key outside
 * [0, T.num_rows) -- PAD slots carry -1 -- gives a row of zero bytes.  This
 * is the lookup of node features, memory, mailbox and edge features for the
 * nodes and edges of a sampled mini-batch (Figure 2, steps 2-3; Section 3).
 * All tables are served by one launch.
 *   nbr        [device] int32[n], or NULL if no table is keyed by node
 *   eid        [device] int64[n], or NULL if no table is keyed by edge
 *   n          slots, >= 0
 *   count      [device] int64 or NULL: when given, only slots
 *              i < min(n, count[0] * per_count) are gathered and the rest of
 *              every output is left untouched (the valid prefix of a hop's
 *              output, whose root count tgl_sample leaves on the device)
 *   per_count  >= 1, slots per counted root
 *   tables     [host] tgl_table[num_tables], num_tables in [1, TGL_MAX_TABLES]
 * Outputs must not overlap the inputs.  Never synchronises.  Errors:
 * TGL_EINVAL for a bad argument, TGL_EDEVICE if the launch fails.
 */
tgl_status tgl_gather(const int32_t *nbr, const int64_t *eid, int64_t n, const int64_t *count,
                      int64_t per_count, const tgl_table *tables, int32_t num_tables, void *stream);

/* ------------------------------------------------------------------------ */
/* Time encoding of sampled slots (Equation 3)                              */
/* ------------------------------------------------------------------------ */

#define TGL_OUT_F32  0     /* float32 output rows                              */
#define TGL_OUT_BF16 1     /* bfloat16 output rows (round to nearest even)    */
#define TGL_MAX_TIME_DIM 4096

/*
 * Time encoding of the slots' time differences (Equation 3, the time encoder
 * of Section 2): out[i][j] = cos(omega[j] * dt[i] + phi[j]) for every slot
 * i < n with dt[i] >= 0; a slot with dt[i] < 0 (PAD slots carry -1) gets a
 * row of zeros.  The argument is formed in double precision (the float
 * product omega * dt is exact there) and reduced modulo 2 pi before a float
 * cosine, so the result is within 1e-6 of the exact value whatever the size
 * of omega * dt (before the bfloat16 rounding, for TGL_OUT_BF16).
 *   dt         [device] float[n] (a hop's dt output)
 *   n          slots, >= 0
 *   count      [device] int64 or NULL: when given, only slots
 *              i < min(n, count[0] * per_count) are encoded and the rest of
 *              `out` is left untouched
 *   per_count  >= 1, slots per counted root
 *   omega, phi [device] float[dim]
 *   dim        in [1, TGL_MAX_TIME_DIM]
 *   out_type   TGL_OUT_F32 or TGL_OUT_BF16
 *   out        [device] n x dim elements of out_type, row-major, 4-byte aligned
 * Never synchronises.  Errors: TGL_EINVAL for a bad argument, TGL_EDEVICE if
 * the launch fails.
 */
tgl_status tgl_time_encode(const float *dt, int64_t n, const int64_t *count, int64_t per_count,
                           const float *omega, const float *phi, int32_t dim, int32_t out_type,
                           void *out, void *stream);

/* ------------------------------------------------------------------------ */
/* Kernel timers (instrumentation for benchmarks)                           */
/* ------------------------------------------------------------------------ */

#define TGL_TIMER_HOP1    0  /* first-hop sampling kernel                     */
#define TGL_TIMER_HOPN    1  /* sampling kernel of hops >= 2                  */
#define TGL_TIMER_COMPACT 2  /* next-hop root compaction (scan + emit)         */
#define TGL_TIMER_BUILD   3  /* whole tgl_tcsr_build                          */
#define TGL_TIMER_GATHER  4  /* tgl_gather                                    */
#define TGL_TIMER_TIMEENC 5  /* tgl_time_encode                               */
#define TGL_TIMER_MFG     6  /* tgl_mfg_export                                */
#define TGL_TIMER_KINDS   7

/*
 * Starts recording HIP events around every kernel of the kinds above, on the
 * stream each is launched on, for up to `capacity` launches (events are
 * created here, so call this outside timed regions).  Resets all totals.
 */
tgl_status tgl_timer_enable(int32_t capacity);

/* Stops recording and releases the events. */
tgl_status tgl_timer_disable(void);

/*
 * Waits for the recorded events and returns, for one kind, the summed
 * duration in milliseconds and the number of launches measured since the
 * last tgl_timer_enable / tgl_timer_reset.
 */
tgl_status tgl_timer_read(int32_t kind, double *total_ms, int64_t *launches);

/* Clears totals and recorded launches (keeps the events). */
tgl_status tgl_timer_reset(void);

/*
 * Records only launches of the kinds whose bit is set in `kinds` (bit k for
 * kind k; all kinds after tgl_timer_enable), so that a timed region carries
 * the events of the kernels it measures and no others.  TGL_EINVAL for bits
 * at or above TGL_TIMER_KINDS.
 */
tgl_status tgl_timer_select(uint32_t kinds);

#ifdef __cplusplus
}
#endif

#endif /* TGL_H */
