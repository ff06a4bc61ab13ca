/*
 * pase.h - C ABI of the MI355X (gfx950) implementation of PaSE's strategy
 * search (V. Elango, "PaSE: Parallelization Strategies for Efficient DNN
 * Training", IPDPS 2021).
 *
 * The library finds a parallelization strategy phi (one configuration per
 * vertex of a computation graph) minimising the cost function F of eq. (1),
 * using the vertex ordering GenerateSeq (Fig. 3) and the dynamic program
 * FindBestStrategy (Fig. 4, recurrence (4)).  The DP tables are filled on the
 * GPU by hand-written HIP kernels; the ordering and the per-vertex plans are
 * computed on the host.
 *
 * Conventions for every function below:
 *  - Return value: PASE_OK (0) or one of the pase_status error codes.  On an
 *    error, caller-owned outputs are left untouched, the handle stays valid
 *    and pase_last_error() describes the problem.
 *  - Pointers named host_* or documented as "host" are host memory; every
 *    array argument is owned by the caller and only read (inputs) or written
 *    (outputs) during the call.  Inputs are copied at pase_graph_create().
 *  - Device memory: the library owns what it allocates (hipMalloc, kept on the
 *    handle and reused across calls) unless the caller lends a device buffer
 *    with pase_set_workspace().
 *  - A handle may be used by one thread at a time.
 *  - Vertex ids are positions in the vertex array passed at creation; edge ids
 *    likewise.  Vertex ids break ties in the vertex ordering (see
 *    pase_enumerate_configs), so they are part of the problem statement.
 */
#ifndef PASE_H
#define PASE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PASE_MAX_DIMS 8   /* loop dims per vertex (iteration-space rank) */
#define PASE_MAX_DEP 8    /* largest dependent set |D(i)| the kernels accept */

typedef enum {
    PASE_OK = 0,
    PASE_ERR_INVALID_ARGUMENT = 1, /* null pointer, ndims not in [1,8], size 0, bad id,
                                      self-loop, tensor-dim map out of range, elems 0,
                                      p not a power of two, array of the wrong length */
    PASE_ERR_NOT_CONNECTED = 2,    /* the graph is not weakly connected (Sec. II) */
    PASE_ERR_BAD_STATE = 3,        /* call order violated (e.g. search before enumeration,
                                      table query without PASE_OPT_KEEP_TABLES) */
    PASE_ERR_OVERFLOW = 4,         /* a cost, or a bound of the costs summed by the
                                      recurrence (a key without its argmin bits), does not fit
                                      in 64 bits; raised by pase_enumerate_configs and
                                      pase_override_costs */
    PASE_ERR_TOO_LARGE = 5,        /* a DP table, |D(i)|, the number of table lookups or
                                      the device memory need exceeds a limit; detected on the
                                      host before any device work */
    PASE_ERR_OUT_OF_MEMORY = 6,    /* a device allocation failed, or a lent workspace is
                                      too small */
    PASE_ERR_HIP = 7,              /* a HIP runtime call failed */
    PASE_ERR_INTERNAL = 8          /* a device-side consistency check failed */
} pase_status;

/* One vertex = one layer and its iteration space (Sec. II).  size[k] is the
 * extent of loop dim k.  reduce_mask bit k marks loop dim k as contracted
 * (splitting it requires a partial-sum reduction).  flops_per_point is the
 * work of one iteration point (2 for a GEMM, 2*kh*kw for a convolution).
 * weight_mask bit k marks loop dim k as an index of the layer's weight tensor,
 * which holds weight_per_point words per point of those dims (kh*kw for a
 * convolution's (co, ci)); 0 = no weights.  Read only with
 * PASE_OPT_GRAD_SYNC.  Convolution geometry, read only with PASE_OPT_HALO:
 * input_mask bit k marks loop dim k as an index of the layer's input tensor
 * ((b, ci, h, w) of a convolution over (b, co, ci, h, w)); halo[k] is the
 * halo width along loop dim k (floor(kernel extent / 2) on a spatial dim, 0
 * elsewhere); a nonzero halo[k] needs bit k of input_mask. */
typedef struct {
    uint32_t ndims;
    uint64_t size[PASE_MAX_DIMS];
    uint32_t reduce_mask;
    uint64_t flops_per_point;
    uint32_t weight_mask;
    uint64_t weight_per_point;
    uint32_t input_mask;
    uint32_t halo[PASE_MAX_DIMS];
} pase_vertex_desc;

/* One edge = a tensor flowing from src to dst (Sec. II).  Tensor dim k is
 * indexed by loop dim src_dim[k] of src and dst_dim[k] of dst (-1: that
 * endpoint does not split tensor dim k).  elems = tensor element count.
 * Parallel edges are allowed; self-loops are not. */
typedef struct {
    uint32_t src, dst, rank;
    int32_t src_dim[PASE_MAX_DIMS];
    int32_t dst_dim[PASE_MAX_DIMS];
    uint64_t elems;
} pase_edge_desc;

/* comm_weight: r, the FLOP-to-byte ratio of eq. (1) (0 selects the default 8).
 * seq_rule: 0 = GenerateSeq where a vertex's d-set never contains itself
 * (default); 1 = the update of Fig. 3 as printed, where an unsequenced vertex
 * may count itself in |v.d|.  Both yield the same minimum cost (Theorem 1) but
 * may order the vertices differently. */
typedef struct {
    uint64_t comm_weight;
    uint32_t seq_rule;
} pase_cost_params;

typedef struct pase_graph_s *pase_graph_t;

typedef enum {
    PASE_OPT_KEEP_TABLES = 1,   /* 1: keep every DP cost table until the next search so that
                                   pase_table_entry / pase_table_fingerprint can read it */
    PASE_OPT_MEMORY_BUDGET = 2, /* bytes of device memory a search may use (default 64 GiB) */
    PASE_OPT_KERNEL = 3,        /* 0 = choose per vertex (default), 1 = generic kernel only */
    PASE_OPT_KEY_TYPE = 4,      /* keys of the fill, cost * 2^ceil(log2 K_v) + c (min and argmin in
                                   one comparison): 0 = choose from the recurrence's cost bounds
                                   (default): fp64 when every key stays within 2^53 (exact integer
                                   arithmetic), else uint64 when within 2^64, else 128-bit keys
                                   (every vertex on prep + the generic kernel); 1 = uint64 unless
                                   the keys need 128 bits; 2 = force 128-bit keys.  Re-plans */
    PASE_OPT_PROFILE = 5,       /* 1: time every fill launch with HIP events (pase_stats);
                                   2: only the row kernel's launches with a column chunk per lane
                                   (the dominant kernel; fewer events, so less overhead) */
    PASE_OPT_SCHEDULE = 6,      /* 5 (default): split chains -- the leaves (dependency level 0)
                                   share their kernel launches on a stream of their own; after
                                   them every row-kernel vertex whose planned fill takes at least
                                   PASE_OPT_BULK_US, with every vertex reading its table, runs on
                                   that stream level by level, and all other vertices level by
                                   level on the caller's stream at the highest wave priority;
                                   events only where a table is read across the two, so the chain
                                   of small vertices and the chain of large fills never wait for
                                   each other level by level.  0: vertices of one dependency level
                                   (whose tables do not read each other) share their kernel
                                   launches, one stream, table memory packed by lifetimes.  1: one
                                   vertex at a time in sequence order (same packing).  4: bulk
                                   lane -- as 5, without the batched leaves (the large fills and
                                   their readers from level 0 on one stream).  4 and 5 keep every
                                   table resident and fall back to 0 over the memory budget.
                                   Other values: INVALID_ARGUMENT */
    PASE_OPT_TILE_COLS = 7,     /* row/column-chunk kernel: columns per lane, 0 = chosen per
                                   vertex (default), else 8, 12, 14, 16, 24 or 28 for every vertex
                                   that kernel runs (a tuning and test knob) */
    PASE_OPT_TILE_ROWS = 8,     /* same kernel: table rows per lane, 0 = chosen (default), 1 or 2 */
    PASE_OPT_TILE_PARTS = 9,    /* same kernel: waves sharing one tile's c range, 0 = chosen
                                   (default), 1, 2 or 4 */
    PASE_OPT_C_SPLITS = 10,     /* same kernel: workgroups sharing one tile's c range (partial
                                   keys reduced by a second launch), 0 = chosen (default), else
                                   min(value, K_v) for every vertex */
    PASE_OPT_CONFIG_SET = 12,   /* configuration set of the next pase_enumerate_configs: 0
                                   (default) power-of-two split factors, p = 2^L <= 65536; 1
                                   every tuple of positive integer factors (Sec. II's C(v)),
                                   1 <= p <= 255 */
    PASE_OPT_ORDER = 13,        /* vertex sequence: 0 (default) GenerateSeq (Fig. 3); 1 the
                                   breadth-first order of Sec. III-A (from vertex 0, neighbours
                                   in ascending id order), on which recurrence (4) is the
                                   breadth-first recurrence (2): every prefix is connected, so
                                   D(i) = D_B(i) and each table reads only its predecessor's.
                                   Re-plans; TOO_LARGE when a dependent set exceeds
                                   PASE_MAX_DEP or a table 2^31 entries (the blow-up that
                                   motivates GenerateSeq) */
    PASE_OPT_TRANSFER = 14,     /* transfer cost model of the next pase_enumerate_configs: 0
                                   (default) split match -- 0 when every tensor dim is split alike
                                   at both ends, else ceil(elems / max(P_u, P_v)); 1 the volume
                                   intersection of Sec. II, max_d |A(v,d)| - |A(v,d) n A(u,d)|
                                   forward plus the same backward, with device d the mixed-radix
                                   point of each configuration's split grid (loop dim 0 slowest)
                                   and each tensor dim cut into equal fractions by the split of
                                   the loop dim it maps to (words rounded up per direction).
                                   Model 1 computes every edge's K_src x K_dst matrix on the
                                   device (workspace grows by 8 bytes per entry); an edge whose
                                   tensor maps several dims to one loop dim is refused
                                   (INVALID_ARGUMENT) when p^(mapped dims) reaches 2^32, and
                                   with distinct mapped loop dims p^2 must stay below 2^32 (p <
                                   65536) */
    PASE_OPT_GRAD_SYNC = 15,    /* 1: the next pase_enumerate_configs adds the data-parallel
                                   weight-gradient all-reduce to every layer cost (an assumed
                                   form; the paper names the communication but prints no
                                   formula): the weight tensor (weight_per_point x the sizes of
                                   the weight_mask dims) is cut into shards by the splits of
                                   those dims, each shard is replicated on the R devices that
                                   differ in the other dims, and a ring all-reduce moves
                                   ceil(2 (R - 1) S / R) words of an S-word shard per device,
                                   weighted by r.  0 (default): the benchmark's cost model */
    PASE_OPT_DIRECT_CELLS = 16, /* vertices with at most this many cells (K_v x table entries)
                                   use the direct fill: every term of recurrence (4) summed per
                                   cell from its source arrays in one launch, no prep blocks --
                                   for the long chains of small dependent vertices, where launch
                                   count dominates.  A level uses it only when all its vertices
                                   qualify (so that it saves launches; any vertex under the
                                   sequential schedule).  Default 2^18; 0 = never.  Not used with
                                   PASE_OPT_KERNEL = 1 */
    PASE_OPT_BULK_US = 17,      /* schedules 4 and 5: planned fill time (microseconds) from which a
                                   row-kernel vertex runs on the bulk stream (default 100) */
    PASE_OPT_FUSED_MIN = 20,    /* 1 (default): a row-kernel vertex without a column digit whose one
                                   lookup is the whole table of its predecessor in the recurrence
                                   (that table's column digit being this vertex, the same row
                                   digits, no outer digits, no c split) has its minimum over c
                                   formed in that predecessor's fill epilogue, combined across
                                   workgroups with 64-bit atomic minima of the packed keys (the
                                   strict "<" tie-break is unchanged: keys are distinct per c),
                                   so the predecessor's table is never written to HBM and read
                                   back; 0: every vertex fills on its own.  Re-plans */
    PASE_OPT_HOIST_ELEMS = 21,  /* one-stream level layout (the level schedule, or the bulk lane
                                   schedule over its memory budget): a vertex whose prep blocks
                                   hold at least this many elements (default 2^20) and read only
                                   tables filled two or more slots before its own has its prep
                                   built on a second stream right after the last of them, while
                                   the slots in between run; its blocks get memory of their own.
                                   0: never.  The allocation-free entry point builds every prep
                                   in its own slot.  Re-plans */
    PASE_OPT_HALO = 19          /* 1: the next pase_enumerate_configs adds the halo exchange of
                                   convolutions to every layer cost (an assumed form; the paper
                                   counts halo communication in t_l but prints no formula): for
                                   every loop dim k with halo[k] > 0 that the configuration
                                   splits, each part receives halo[k] boundary rows of the input
                                   from each of its two neighbours along k, a row being the
                                   part's share of the input tensor over its other dims:
                                   2 * halo[k] * ceil(prod_{j in input, j != k} n_j /
                                   prod_{j in input, j != k} s_j) words, weighted by r.
                                   0 (default): the benchmark's cost model */
} pase_option;

/* Search statistics of the last pase_find_best_strategy call. */
typedef struct {
    uint64_t cells;            /* DP cell updates: sum over vertices of K_i * |table i| */
    uint64_t table_entries;    /* sum of |table i| */
    uint64_t workspace_bytes;  /* device bytes the search used */
    uint32_t max_dep;          /* max |D(i)| */
    uint32_t key_type;         /* 0 = fp64 exact-integer keys, 1 = uint64 keys */
    uint32_t launches;         /* kernels launched by the search */
    uint32_t rows_vertices;    /* vertices filled by the row/column-chunk kernel */
    uint64_t rows_cells;       /* cells filled by that kernel */
    double host_plan_ms;       /* pase_enumerate_configs (host): seq_ms + plan_ms */
    double wall_ms;            /* pase_find_best_strategy, host wall clock */
    double fill_ms;            /* PASE_OPT_PROFILE: sum of the timed fill launches' event times
                                  (profile 2: the column-form row-kernel launches only) */
    double rows_fill_ms;       /* PASE_OPT_PROFILE: same, row/column-chunk kernel only */
    uint32_t rows_launches;    /* PASE_OPT_PROFILE: launches of that kernel */
    uint32_t slots;            /* launch slots: dependency levels, or vertices when sequential */
    uint64_t stream_cells;     /* cells of the row kernel's column-less (streaming) form, a part
                                  of rows_cells */
    double stream_fill_ms;     /* PASE_OPT_PROFILE: event time of those launches, a part of
                                  rows_fill_ms */
    uint32_t stream_launches;  /* PASE_OPT_PROFILE: their launches, a part of rows_launches */
    uint32_t schedule;         /* schedule the search ran with (PASE_OPT_SCHEDULE values) */
    uint32_t pad0;
    /* phases of the last enumeration and search, milliseconds */
    double seq_ms;             /* pase_enumerate_configs, host: GenerateSeq and the sets D(i), X(i), S(i) */
    double plan_ms;            /* pase_enumerate_configs, host: kernel plans and the device memory layout */
    double setup_ms;           /* pase_find_best_strategy, host: key bound, launch descriptors and the
                                  constant-region image, up to the upload */
    double cost_tables_ms;     /* PASE_OPT_PROFILE, device: upload and cost-table kernels */
    double fill_span_ms;       /* PASE_OPT_PROFILE, device: from the end of the cost tables to the end
                                  of the last fill or split reduction (every prep, fill and reduction
                                  launch and the gaps between them) */
    double backtrack_ms;       /* PASE_OPT_PROFILE, device: back-substitution */
    double assign_ms;          /* pase_assign_devices, host: the last device assignment */
} pase_run_stats;

/* Copy a computation graph G=(V,E) (Sec. II) into a new handle.
 * v: host array of nv vertices; e: host array of ne edges; params: NULL for
 * defaults.  Errors: INVALID_ARGUMENT, NOT_CONNECTED. */
pase_status pase_graph_create(const pase_vertex_desc *v, uint32_t nv, const pase_edge_desc *e,
                              uint32_t ne, const pase_cost_params *params, pase_graph_t *out);

/* Release the handle and every device buffer it owns.  NULL is ignored. */
void pase_graph_destroy(pase_graph_t g);

/* Text of the last error on this handle ("" if none).  Valid until the next call. */
const char *pase_last_error(pase_graph_t g);

/* Enumerate the configuration set C(v) of every vertex for p modeled devices
 * (Sec. II: tuples of split factors with product <= p): by default the
 * power-of-two factors, p = 2^L with L <= 16; with PASE_OPT_CONFIG_SET = 1
 * every positive integer factor, 1 <= p <= 255.  Configurations are ordered
 * lexicographically by the split tuple with loop dim 0 slowest (for powers of
 * two the same order as the exponent tuple).  Then order the vertices with
 * GenerateSeq (Fig. 3; ties of |u.d| go to the lowest vertex id), derive the
 * dependent sets D(i), connected sets X(i) and connected subsets S(i)
 * (Sec. III-B) and the device memory plan.  Host only; resets any earlier
 * search state and cost override.
 * Errors: INVALID_ARGUMENT (p), OVERFLOW (a layer or transfer cost, or a
 * bound of a sum of them along the recurrence, exceeds 64 bits), TOO_LARGE
 * (|D(i)| > PASE_MAX_DEP, a table over 2^31 entries, K_v > 65535). */
pase_status pase_enumerate_configs(pase_graph_t g, uint32_t p);

/* K_v = |C(v)|.  Needs pase_enumerate_configs. */
pase_status pase_num_configs(pase_graph_t g, uint32_t v, uint32_t *k);

/* Split factors of configuration idx of vertex v into host array splits[ndims]. */
pase_status pase_config_splits(pase_graph_t g, uint32_t v, uint32_t idx, uint32_t *splits);

/* The GenerateSeq order: order[i] = vertex id at position i (host array of nv). */
pase_status pase_get_sequence(pase_graph_t g, uint32_t *order);

/* D(v) of vertex id v (Sec. III-B), ascending vertex ids, into host out[cap];
 * *n receives |D(v)| (TOO_LARGE if cap < |D(v)|). */
pase_status pase_get_dependent_set(pase_graph_t g, uint32_t v, uint32_t *out, uint32_t cap,
                                   uint32_t *n);

/* Set one pase_option. */
pase_status pase_set_option(pase_graph_t g, pase_option opt, uint64_t value);

/* Replace the cost model by caller-given costs (testing hook; needs
 * pase_enumerate_configs).  layer: host array, the K_v layer costs of every
 * vertex concatenated in vertex order.  edge: host array, for every edge the
 * row-major K_src x K_dst matrix of r*t_x, concatenated in edge order (may be
 * NULL when ne = 0).  Re-plans the key type (R10).  Cleared by the next
 * pase_enumerate_configs.  Errors: OVERFLOW (a bound of the costs summed by
 * the recurrence exceeds 64 bits; the earlier costs stay in force). */
pase_status pase_override_costs(pase_graph_t g, const uint64_t *layer, const uint64_t *edge);

/* Device bytes pase_find_best_strategy needs (after pase_enumerate_configs). */
pase_status pase_workspace_size(pase_graph_t g, uint64_t *bytes);

/* Lend a device buffer of `bytes` bytes (256-byte aligned) for the next
 * searches instead of library allocations; NULL returns to library-owned
 * memory.  The caller keeps ownership and must keep it alive while the handle
 * uses it. */
pase_status pase_set_workspace(pase_graph_t g, void *device_ptr, uint64_t bytes);

/* Run FindBestStrategy (Fig. 4) on the GPU: cost tables, per-vertex DP table
 * fill in sequence order, and back-substitution from the last vertex.
 * stream: a hipStream_t (NULL = the null stream) on the current device; all
 * device work is enqueued on it and the call returns after it is finished.
 * min_cost: host, receives R(|V|, {}) = min over phi of F(G, phi) (Theorem 1).
 * config_idx: host array of nv, receives the chosen configuration index per
 * vertex id.  Among equal-cost configurations a table entry keeps the lowest
 * index (the strict "<" of Fig. 4 with ascending indices).
 * Errors: BAD_STATE, TOO_LARGE, OUT_OF_MEMORY, HIP, INTERNAL. */
pase_status pase_find_best_strategy(pase_graph_t g, void *stream, uint64_t *min_cost,
                                    uint32_t *config_idx);

/* Allocation-free variant of pase_find_best_strategy, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  It allocates nothing -- no hipMalloc,
 * hipFree, pinned host memory, stream or event: every device buffer of the
 * search (constant region, DP and argmin tables, prep blocks, split scratch)
 * lives in one static device array of PASE_NOALLOC_WORKSPACE_BYTES that each
 * GPU the library runs on holds until the process ends, and the constant
 * region is staged through a static host buffer of the same size.  Same
 * arguments, results and errors as pase_find_best_strategy, plus TOO_LARGE
 * when pase_workspace_size() exceeds PASE_NOALLOC_WORKSPACE_BYTES (checked on
 * the host before any device work).  Profiling (PASE_OPT_PROFILE) is ignored
 * and a two-stream plan (PASE_OPT_SCHEDULE 4 or 5) runs level by level on `stream`.
 * The array keeps the last call's contents and every call on one GPU shares
 * it: calls in one process are serialized by a lock, calls from different
 * processes that overlap on one GPU race, and the next allocation-free search
 * on that GPU (any handle) overwrites the tables that pase_table_entry /
 * pase_table_fingerprint read after this one. */
#define PASE_NOALLOC_WORKSPACE_BYTES (64ull << 20)
pase_status pase_find_best_strategy_noalloc(pase_graph_t g, void *stream, uint64_t *min_cost,
                                            uint32_t *config_idx);

/* Read entry T_v[dep_cfg] of the DP table of vertex v and its argmin after a
 * search with PASE_OPT_KEEP_TABLES=1.  dep_cfg: host array of |D(v)|
 * configuration indices, one per member of D(v) in ascending vertex id. */
pase_status pase_table_entry(pase_graph_t g, uint32_t v, const uint32_t *dep_cfg, uint64_t *cost,
                             uint32_t *argmin);

/* Order-independent fingerprints of the DP table of vertex v (needs
 * PASE_OPT_KEEP_TABLES=1): with phi the canonical index (D(v) ascending,
 * first digit slowest) and mix the SplitMix64 output function,
 *   fp_cost = sum_phi mix(mix(phi) ^ T[phi]),  fp_arg = sum_phi mix(mix(phi) ^ A[phi])
 * (sums mod 2^64). */
pase_status pase_table_fingerprint(pase_graph_t g, uint32_t v, uint64_t *fp_cost, uint64_t *fp_arg);

/* Device-computed layer costs t_l(v, c) of the last search, host out[K_v]. */
pase_status pase_layer_costs(pase_graph_t g, uint32_t v, uint64_t *out);

/* Device-computed r*t_x(e, c_src, c_dst) of edge e, host out[K_src*K_dst]
 * row-major (evaluated on the GPU from the configurations). */
pase_status pase_edge_costs(pase_graph_t g, uint32_t e, uint64_t *out);

/* Statistics of the last search. */
pase_status pase_stats(pase_graph_t g, pase_run_stats *out);

/* Plan of one vertex (after pase_enumerate_configs) and, after a search with
 * PASE_OPT_PROFILE=1, its fill time. */
typedef struct {
    uint32_t position;   /* index in the GenerateSeq order */
    uint32_t kernel;     /* 0 = generic fill, 1 = row/column-chunk fill, 2 = direct fill */
    uint32_t num_configs, dep_count;
    uint64_t entries;    /* |table| = product of K over D(v) */
    uint64_t cells;      /* K_v * entries */
    int32_t column;      /* row kernel: column digit (vertex id), -1 for none or the generic kernel */
    uint32_t outer, rows, tile_cols;
    uint32_t tile_rows;  /* rows per lane (1 or 2) */
    uint32_t splits, row_terms, lookups;
    uint32_t parts;      /* row kernel: waves sharing one tile's c range (1, 2 or 4) */
    double fill_ms;      /* PASE_OPT_PROFILE: event time of this vertex's fill kernel */
    uint32_t level;      /* dependency level: 1 + the largest level of the tables it reads */
    uint32_t lane;       /* bulk lane schedule: the stream it runs on: 0 = the caller's (small vertices,
                            highest wave priority), 1 = the bulk stream (large fills and their readers) */
    uint64_t key_bound;  /* upper bound of every summed cost before the min over c (keys stay
                            below (key_bound + 1) * 2^ceil(log2 K_v)); ~0 if it exceeds 64 bits */
    uint64_t table_bound; /* upper bound of every entry of its DP table; ~0 likewise */
    uint32_t key_type;    /* key type of the plan (the same for every vertex): 0 fp64, 1 uint64, 2 128-bit */
    uint32_t fused;       /* PASE_OPT_FUSED_MIN: 1 = its fill also forms the minimum of its table's reader,
                             2 = that reader (its fill is then a one-split reduction of those keys), 0 = neither */
    int32_t prep_after;   /* its prep blocks read only tables of slots up to this one (-1: none) and are
                             built right after it, beside the launches of the slots in between -- on a
                             side stream (level layout) or at the end of that slot's launches on lane
                             prep_lane (schedules 4 and 5); -2 = built in its own slot */
    uint32_t prep_lane;   /* schedules 4 and 5, prep_after >= 0: the lane its prep runs on (that of the
                             tables it reads) */
} pase_vertex_info;

pase_status pase_vertex_info_get(pase_graph_t g, uint32_t v, pase_vertex_info *out);

/* Device assignment of a strategy (Sec. II, the paragraph on assigning
 * devices after the search): the cost model numbers the parts of each
 * configuration by their grid point; this places them on the p modeled
 * devices greedily so that tensors stay where they are.  Vertices in
 * ascending id order; vertex 0 puts part g on device g; every later vertex v
 * places all its parts on distinct devices, pair (part q, device d) by pair,
 * largest locality first, ties to the lower part and then the lower device,
 * where the locality of (q, d) is the number of tensor elements, over all
 * edges joining v to an already placed (lower-id) vertex u, that part q and
 * u's part on d both cover.  Part geometry: loop dim k of a configuration is
 * cut into s_k equal fractions, part g is the mixed-radix grid point of g
 * (loop dim 0 slowest), a tensor dim covers the fraction of the loop dim it
 * maps to (all of it when unmapped); shared elements of two parts are
 * floor(elems * shared fraction).  Host only, after pase_enumerate_configs.
 * config_idx: host array of nv configuration indices (a strategy, e.g. from
 * pase_find_best_strategy).  devices: host array of nv * p, receives the part
 * of vertex v on device d at [v * p + d], -1 where v has no part.
 * edge_locality (host array of ne, or NULL): the elements of each edge's
 * tensor the two ends hold on the same device, summed over devices.
 * edge_xfer (host array of ne, or NULL): r * t_x of each edge under this
 * assignment -- the volume model of PASE_OPT_TRANSFER = 1 with these devices
 * in place of the grid numbering (equal to it when both ends keep the grid
 * numbering).  Errors: INVALID_ARGUMENT (null array, index out of range),
 * BAD_STATE (no enumeration), TOO_LARGE (p > 1024, or an edge cut into 2^64
 * cells or more), OVERFLOW (the tensor elements of one vertex's edges, or a
 * transfer cost, exceed 64 bits). */
pase_status pase_assign_devices(pase_graph_t g, const uint32_t *config_idx, int32_t *devices,
                                uint64_t *edge_locality, uint64_t *edge_xfer);

/* Diagnostics (host only, no device work): build the kernel descriptors,
 * batched launches and constant-region image that pase_find_best_strategy
 * would upload for the current plan and costs, against a stand-in workspace
 * address, into a host buffer of exactly the constant region's size, and
 * check that every vertex is filled by exactly one launch.  *image_bytes
 * receives that size.  Errors: BAD_STATE (no plan), INTERNAL (a region or
 * table bound of the plan would be exceeded), TOO_LARGE (a launch grid). */
pase_status pase_plan_check(pase_graph_t g, uint64_t *image_bytes);

#ifdef __cplusplus
}
#endif

#endif /* PASE_H */
