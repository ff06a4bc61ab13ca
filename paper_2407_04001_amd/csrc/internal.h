// Internal data structures of libpase (host planning + device descriptors).
//
// Vocabulary (Sec. III-B of the paper): the vertices are visited in the order
// of GenerateSeq; position i holds vertex v_i with dependent set D(i).  The DP
// table of position i, T_i, has one entry per assignment phi of D(i); the
// entry is min over the configurations c of v_i of
//     layer cost + transfer costs to later neighbours + sum_j T_j[phi' | D(j)]
// (recurrence (4)).  Here the terms of that sum are grouped by the digits of
// phi they depend on, and the "digits" of a table are the members of its
// dependent set in the table's own memory order.
#pragma once

#include <array>
#include <cstdint>
#include <string>
#include <vector>

#include "pase.h"

namespace pase {

constexpr int kMaxDims = PASE_MAX_DIMS;
constexpr int kMaxDep = PASE_MAX_DEP;
constexpr int kMaxATerms = 4;      // per-lane row terms of the row kernel
constexpr int kMaxGTerms = 24;     // terms of the generic kernel
constexpr int kMaxContrib = 64;    // contributions to one precomputed block
constexpr int kMaxBlocks = kMaxDep + 1;
constexpr uint64_t kMaxTableEntries = (1ull << 31) - 1;
constexpr uint32_t kAssignMaxDevices = 1024;   // p bound of the device assignment

// ------------------------------------------------------------------ device descriptors
struct DevVertex {            // configuration data of one vertex (uploaded once per search)
    uint64_t ex_off;          // byte offset of its split rows (K x ndims uint8)
    uint64_t L_off;           // element offset of its layer-cost vector
    uint64_t flops;           // flops_per_point * prod(size)
    uint64_t keep_n;          // prod of the sizes of the non-contracted dims
    uint32_t K, ndims, reduce_mask;
    uint32_t factors;         // 0: split rows hold log2 of power-of-two factors and the
                              // per-configuration device byte its exponent sum; 1: both
                              // hold the factors / device count themselves (p <= 255)
    uint64_t weight_n;        // gradient term: words of the weight tensor (0: no term)
    uint32_t weight_mask;
    uint32_t halo_mask;       // halo term: loop dims with a halo (0: no term)
    uint32_t input_mask;      // halo term: loop dims indexing the input tensor
    uint32_t halo_w[kMaxDims];   // halo width per loop dim
    uint64_t halo_n[kMaxDims];   // halo term: prod of the input dims' sizes other than this one
};

struct DevEdge {
    uint32_t src, dst, rank;
    uint32_t factors;         // as DevVertex::factors
    int8_t sdim[kMaxDims], ddim[kMaxDims];
    uint64_t elems;
    uint64_t sig_off;         // element offset of its split signatures: K_src, then K_dst
    uint64_t mat_off;         // volume transfer model: element offset of its K_src x K_dst matrix
    uint64_t row0;            // volume transfer model: its first matrix row among all edges' rows
};

// One contribution to a precomputed block element (see Prep below).
enum ContribKind : uint32_t { kContribLayer = 0, kContribEdge = 1, kContribTable = 2 };
struct Contrib {
    uint32_t kind;
    uint32_t edge;            // kContribEdge: edge id
    uint32_t dig;             // kContribEdge: plan digit of the other endpoint
    uint32_t vi_is_src;       // kContribEdge: v_i is the edge's source
    const void *ptr;          // kContribTable: value table (key type's value form, or uint64 for
                              // caller-given edge matrices)
    uint32_t sc;              // kContribTable: element stride of v_i's configuration
    uint32_t raw_u64;         // kContribTable: 1 = plain uint64 costs (caller-given edge
                              // matrices), 0 = a DP table already in this vertex's key space
    uint32_t sd[kMaxDep];     // kContribTable: element stride per plan digit (0 = unused)
};

// A precomputed block: a key-space array over (pre digits, c, post digit)
// laid out [pre...][c][ld].  Each element is the sum of its contributions,
// multiplied by 2^bits (the low bits of a key hold the configuration index).
struct Block {
    uint64_t out_off;         // element offset in the block scratch
    uint64_t elems;           // prod(pre radices) * K * ld
    uint32_t npre;
    uint32_t pre[kMaxDep];    // plan digits, slowest first
    uint32_t prerad[kMaxDep];
    int32_t post;             // plan digit, -1 = none
    uint32_t postrad;         // its radix (columns actually filled)
    uint32_t ld;              // row pitch (>= postrad, padded columns hold 0)
    uint32_t c_begin, c_end;  // contribution range
    uint32_t rows;            // prod(pre radices)
    uint32_t chunks;          // workgroups per row: ceil(K * ld / (kPrepThreads * span))
    uint32_t wg_begin;        // first workgroup of this block
    uint32_t span;            // kPrepThreads-element spans per workgroup
};

constexpr uint32_t kPrepThreads = 256;

struct PrepArgs {
    uint32_t vi, K, bits, nblocks;
    uint64_t total;           // sum of block elements
    uint32_t nwg, pad;        // workgroups of this vertex
    void *blocks;             // this vertex's block scratch
    Block blk[kMaxBlocks];
};

// One vertex of a batched launch: its descriptor index (sequence position)
// and its first workgroup.  The workgroups of a launch are the concatenation
// of the workgroups of its vertices.
struct BatchEntry {
    uint32_t pos;
    uint32_t first;
    uint32_t prio;            // 1: the bulk lane schedule's small vertices -- their waves issue first
    uint32_t kind;            // row-kernel launches: 0 a row fill, 1 a two-term generic fill riding along
};
constexpr uint32_t kEntryGeneric2 = 1;

struct ATerm {                // per-lane row term of the row kernel (key space)
    const void *ptr;
    uint32_t sc;              // stride of c
    uint32_t bytes;           // size of the array (buffer-load range, < 2^31)
    uint32_t sdO[kMaxDep];    // strides per outer digit
    uint32_t sdR[kMaxDep];    // strides per row digit
};

struct RowsArgs {
    const void *B;            // [o][c][ldz] key space: layer cost, c, outer and column terms
    uint32_t ldz, Kz, K, bits;
    uint32_t MO, MR, tiles_per_o, nchunks;
    uint32_t nsplit, cper;
    uint32_t nO, nR;
    uint32_t radO[kMaxDep], radR[kMaxDep];
    uint32_t na;
    ATerm a[kMaxATerms];
    void *T;                  // output values, index z*(MO*MR) + o*MR + r
    uint16_t *A;              // output argmins
    void *partial;            // nsplit > 1: keys [split][N]
    uint64_t N;
    uint64_t total_tiles;     // tiles (a workgroup takes 4 / parts of them)
    uint32_t nblocks_launched;
    uint32_t parts;           // waves sharing one tile's c range: 1, 2 or 4
    uint32_t out_shift;       // bits of the table's reader: values are stored x 2^out_shift
    // Fused minimum of the reader (fz_keys non-null): the table's only reader
    // v_j is this vertex's column digit and takes, per row r, the minimum over
    // its configuration c = z of T[z][r] plus its other row terms at (r, z)
    // plus its column block at z.  The epilogue forms those keys of v_j for
    // the tile's columns and min-combines them into fz_keys[r] atomically (64-bit
    // keys, non-negative, so their bit patterns order like the keys); a
    // one-split reduction then turns the keys into v_j's table.  T may then
    // be null: nothing else reads it.
    void *fz_keys;
    const void *fz_B;         // the reader's column block, element z * fz_ldz
    uint32_t fz_ldz, fz_na;   // its row pitch; the reader's row terms other than T
    ATerm fz_a[kMaxATerms];   // those row terms (ptr, sc, sdR over the same row digits)
};

struct GTerm {                // term of the generic kernel (key space)
    const void *ptr;
    uint32_t sc, pad;
    uint32_t sd[kMaxDep];
};

struct GenericArgs {
    uint32_t m, K, bits, nt;
    uint32_t group_log2;      // lanes per entry = 2^group_log2 (c is strided over them)
    uint32_t pad2;
    uint32_t rad[kMaxDep];    // radices of the plan digits (= T_i layout), slowest first
    GTerm t[kMaxGTerms];
    void *T;
    uint16_t *A;
    uint64_t N;
    uint32_t out_shift, nblk;  // nblk: workgroups of this vertex
};

// Direct fill of a small vertex: every term of recurrence (4) -- layer cost,
// transfer costs, table lookups -- is summed per (entry, c) from its source
// arrays (contributions [c_begin, c_end) over the plan digits), with no prep
// blocks; one launch per level instead of prep + fill (+ split reduction).
struct DirectArgs {
    uint32_t vi, K, bits, out_shift;
    uint32_t m;               // plan digits (= T_i layout), slowest first
    uint32_t group_log2;      // lanes per entry = 2^group_log2 <= 256 (c is strided over them)
    uint32_t c_begin, c_end;  // contributions
    uint32_t rad[kMaxDep];
    uint32_t nblk, pad;       // nblk: workgroups of this vertex
    uint64_t N;
    void *T;
    uint16_t *A;
};

struct ReduceArgs {
    const void *partial;
    void *T;
    uint16_t *A;
    uint64_t N;
    uint32_t nsplit, bits, out_shift, nblk;
};

struct BacktrackDesc {        // per position, for the back-substitution kernel
    const uint16_t *A;
    uint32_t vi, m;
    uint32_t level;           // backward level: 1 + max level over D(i) (0 when D(i) is empty)
    uint32_t K;               // configurations of v_i: a stored argmin must be below it
    uint32_t dig[kMaxDep];    // vertex ids of the layout digits
    uint64_t stride[kMaxDep];
};

constexpr uint32_t kMaxBacktrackThreads = 1024;   // one thread per position

struct SearchOut {            // written by the back-substitution kernel
    uint64_t min_cost;
    uint32_t status;          // 0 = ok; 4 = an argmin out of range
    uint32_t pad;
};

// PASE_OPT_SCHEDULE values
enum SchedKind { kSchedLevel = 0, kSchedSeq = 1, kSchedBulk = 4, kSchedSplit = 5 };
constexpr int kSplitBatchedLevels = 1;   // split chains: levels that stay batched on one lane

// ------------------------------------------------------------------ host plan
struct TermRef {
    int j;                    // position of the producer (last vertex of the component)
    std::vector<int> dig;     // D(j) - {v_i}: vertex ids
};

enum KernelKind { kGeneric = 0, kRows = 1, kDirect = 2 };

struct VPlan {
    int vi = -1;
    uint32_t K = 0, bits = 0;
    std::vector<int> D;             // D(i), ascending vertex id
    std::vector<int> layout;        // plan digits = T_i memory order, slowest first (vertex ids)
    std::vector<uint64_t> stride;   // element stride of each layout digit in T_i
    uint64_t N = 1;
    std::vector<int> edges;         // edges joining v_i and a later vertex
    std::vector<TermRef> terms;     // one lookup per connected subset in S(i)
    int consumer = -1;              // position whose lookups read T_i
    uint32_t out_shift = 0;         // T_i is stored x 2^(bits of its reader): in the reader's key space
    KernelKind kernel = kGeneric;
    // row kernel shape
    int z = -1;                     // column digit (vertex id)
    std::vector<int> O, R;          // outer / row digits (vertex ids), slowest first
    uint32_t TZ = 0, TM = 1, ldz = 0, nchunks = 0, nsplit = 1, cper = 0, parts = 1;
    uint64_t MO = 1, MR = 1;
    uint32_t na = 0;                // row kernel: per-lane row terms
    // fused minimum (row kernel): this vertex's table feeds only the minimum
    // of its column digit's vertex, which its fill forms in the epilogue
    int fuse_into = -1;             // position of that reader, -1 = none
    int fused_from = -1;            // the reader: position of the producer, -1 = none
    uint64_t fkeys_off = 0;         // the reader: bytes into the fused-key region
    // hoisted prep: the blocks read only tables filled by slot prep_after or
    // earlier, so they are built right after that slot, beside the slots in
    // between -- on a side stream (level layout), or at the end of that
    // slot's group of lane prep_lane (lanes); -2 = not hoisted
    int prep_after = -2;
    int prep_lane = 0;
    double fill_ms = 0;             // last profiled fill time
    double est_us = 0;              // planned fill time (tile model), for the schedule
    // memory
    uint64_t T_off = 0, A_off = 0;  // bytes into the table arenas
    uint64_t block_elems = 0;       // block scratch this vertex needs
    uint64_t block_off = 0;         // bytes into the block scratch
    uint64_t partial_off = 0;       // bytes into the split scratch
    // schedule
    int level = 0;                  // dependency level: 1 + max level of the tables it reads
    int slot = 0;                   // launch slot: its level (level schedule) or its position
    int lane = 0;                   // bulk lane schedule: 0 = the caller's stream (small vertices, level
                                    // by level), 1 = the bulk stream (the large fills and their readers)
};

struct Plan {
    std::vector<int> seq, pos;
    std::vector<VPlan> v;           // by position
    uint64_t cells = 0, entries = 0, rows_cells = 0, stream_cells = 0;
    uint32_t max_dep = 0, rows_vertices = 0;
    // workspace layout, byte offsets from the workspace base
    uint64_t off_ex = 0, off_vert = 0, off_edge = 0, off_L = 0, off_lsum = 0, off_sig = 0,
             off_ovedge = 0, off_contrib = 0,
             off_bt = 0, off_zero = 0, off_cfg = 0, off_out = 0, off_vmat = 0, off_T = 0, off_A = 0, off_block = 0,
             off_partial = 0, off_fused = 0, total = 0;
    uint64_t T_bytes = 0, A_bytes = 0, block_bytes = 0, partial_bytes = 0, contrib_count = 0;
    uint64_t fused_bytes = 0;       // keys of the fused minima (initialised by k_cost_tables)
    uint32_t hoisted = 0;           // vertices whose prep runs on the side stream
    uint32_t fused = 0;             // fused producer/reader pairs
    uint64_t sig_count = 0;         // split signatures of all edge endpoints
    int nslots = 0;                 // launch slots (levels, or positions when sequential)
    bool by_level = false;          // the vertices of one dependency level share launches
    bool resident = false;          // every table and scratch buffer resident at once (no reuse)
    uint64_t off_desc = 0, off_batch = 0;   // per-vertex launch descriptors, batch tables
};

struct DeviceState;   // defined by the device runtime

}  // namespace pase

struct pase_graph_s {
    std::vector<pase_vertex_desc> V;
    std::vector<pase_edge_desc> E;
    uint64_t r = 8;
    uint32_t seq_rule = 0;
    std::vector<std::vector<int>> nbr;     // undirected, deduplicated, ascending
    std::string err;
    // options
    bool keep_tables = false;
    int profile = 0;                // pase_option PASE_OPT_PROFILE: 0 off, 1 every fill launch, 2 the
                                    // column-form row-kernel launches only
    uint64_t mem_budget = 64ull << 30;
    int kernel_mode = 0, key_mode = 0;
    uint32_t tile_cols = 0, tile_rows = 0, tile_parts = 0, c_splits = 0;   // 0 = chosen by the plan
    int schedule = pase::kSchedSplit;   // pase_option PASE_OPT_SCHEDULE (SchedKind)
    int order_mode = 0;             // pase_option PASE_OPT_ORDER: 0 GenerateSeq, 1 breadth-first
    // configurations
    bool enumerated = false;
    uint32_t config_set = 0;        // pase_option PASE_OPT_CONFIG_SET, read by pase_enumerate_configs
    uint32_t transfer_opt = 0;      // pase_option PASE_OPT_TRANSFER, read by pase_enumerate_configs
    uint32_t grad_opt = 0;          // pase_option PASE_OPT_GRAD_SYNC, read by pase_enumerate_configs
    uint32_t halo_opt = 0;          // pase_option PASE_OPT_HALO, read by pase_enumerate_configs
    bool halo = false;              // the enumerated layer costs carry the halo term
    std::vector<std::array<uint64_t, pase::kMaxDims>> halo_n;   // halo term: per vertex and loop dim, the
                                    // product of the input dims' sizes other than that dim
    uint64_t direct_cells = 1ull << 18;  // pase_option PASE_OPT_DIRECT_CELLS
    uint32_t bulk_us = 100;         // pase_option PASE_OPT_BULK_US
    bool fuse_min = true;           // pase_option PASE_OPT_FUSED_MIN
    uint64_t hoist_elems = 1ull << 20;   // pase_option PASE_OPT_HOIST_ELEMS (0 = never)
    std::vector<uint64_t> weight_n; // gradient term of the enumeration: weight words per vertex (0 = none)
    bool volume = false;            // the enumerated transfer model is the volume intersection
    std::vector<uint64_t> mat_off;  // volume model: element offset of each edge's cost matrix
    uint64_t mat_total = 0;         // volume model: entries of all edge matrices
    std::vector<uint64_t> mat_row0; // volume model: first matrix row of each edge (rows = K_src)
    uint64_t mat_rows = 0;          // volume model: rows of all edge matrices
    uint32_t p = 0;
    bool factors = false;           // the enumerated set: split rows hold factors, not exponents
    std::vector<uint32_t> K;
    // the configurations of a vertex depend only on its dimension count: one
    // row set per count, ex_rows[d][c*d + k] = log2 of the split factor, or the
    // factor itself when `factors`
    std::vector<std::vector<uint8_t>> ex_rows;
    std::vector<const std::vector<uint8_t> *> ex;  // [v] -> ex_rows[ndims of v]
    std::vector<uint64_t> flops, keep_n;
    std::vector<uint64_t> maxL;            // upper bound of the layer cost per vertex
    std::vector<uint64_t> maxR;            // upper bound of the transfer cost per edge
    // caller-given costs
    bool overridden = false;
    std::vector<uint64_t> ov_layer, ov_edge, ov_layer_off, ov_edge_off;
    // plan
    pase::Plan plan;
    bool planned = false;
    // keys of the plan (R10): 0 fp64, 1 uint64, 2 128-bit (packed keys past 2^64 while every
    // cost sum fits 64 bits; such a plan runs every vertex on prep + the generic kernel)
    uint32_t plan_key_type = 0;
    bool plan_wide = false;         // the plan was built for 128-bit keys
    // last search
    bool searched = false;
    uint32_t key_type = 0;
    pase_run_stats stats{};
    // a workspace lent by the caller (pase_set_workspace), else library-owned memory
    void *lent_ws = nullptr;
    uint64_t lent_bytes = 0;
    // device runtime
    pase::DeviceState *dev = nullptr;
};

namespace pase {
// host.cpp
pase_status fail(pase_graph_t g, pase_status st, const std::string &msg);
uint32_t choose_key_type(pase_graph_t g, pase_status *st);
uint32_t key_bytes(pase_graph_t g);   // bytes of a table value / block key of the plan (8 or 16)
// launch_plan.cpp: the launch descriptors and constant image of the plan's key
// type, built against a stand-in workspace base into a host buffer of exactly
// the constant region's size (no device work)
pase_status plan_check(pase_graph_t g, uint64_t *image_bytes);
// device.hip
void device_release(pase_graph_t g);
pase_status device_search(pase_graph_t g, void *stream, uint64_t *min_cost, uint32_t *cfg);
pase_status device_search_noalloc(pase_graph_t g, void *stream, uint64_t *min_cost, uint32_t *cfg);
pase_status device_table_entry(pase_graph_t g, int pos, uint64_t idx, uint64_t *cost,
                               uint32_t *arg);
pase_status device_fingerprint(pase_graph_t g, int pos, uint64_t *fpT, uint64_t *fpA);
pase_status device_layer_costs(pase_graph_t g, uint32_t v, uint64_t *out);
pase_status device_edge_costs(pase_graph_t g, uint32_t e, uint64_t *out);
}  // namespace pase
