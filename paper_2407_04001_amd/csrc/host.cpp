// Host side of libpase: graph validation, configuration enumeration, the
// GenerateSeq vertex order (Fig. 3), connected sets / dependent sets /
// connected subsets (Sec. III-B), per-vertex DP plans and the device memory
// layout.  No HIP calls here: everything is pure host computation so it can be
// exercised without a GPU.
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>
#include <numeric>
#include <unordered_map>

#include "internal.h"

using namespace pase;

namespace pase {

pase_status fail(pase_graph_t g, pase_status st, const std::string &msg) {
    if (g) g->err = msg;
    return st;
}

static bool mul_ok(uint64_t a, uint64_t b, uint64_t *out) { return !__builtin_mul_overflow(a, b, out); }
static bool add_ok(uint64_t a, uint64_t b, uint64_t *out) { return !__builtin_add_overflow(a, b, out); }
static uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }
static uint32_t bits_for(uint32_t K) {
    uint32_t b = 0;
    while ((1u << b) < K) b++;
    return b;
}

// Upper bounds of the DP quantities at every sequence position i, used to
// size the keys.  Q_i(phi, c) -- the layer cost of v_i at c, plus r * t_x of
// every edge joining v_i and a later vertex, plus the table lookup of every
// connected subset -- is at most maxL(v_i) + sum maxR + sum Tmax_j.  The table
// entry T_i(phi) = min_c Q_i(phi, c) is at most Q_i(phi, c0) for any single c0:
// with model costs c0 is the cheapest of the unsplit configuration (cost F)
// and the ones that split a single dim p ways (costs evaluated exactly); with
// caller-given costs it is the cheapest layer configuration.  These bounds
// follow the recurrence instead of summing every cost of the graph, so deep
// graphs keep exact fp64 keys.  false: a bound exceeds 64 bits.
bool cost_bounds(pase_graph_t g, std::vector<uint64_t> *qmax, std::vector<uint64_t> *tmax) {
    const Plan &P = g->plan;
    const size_t n = P.v.size();
    qmax->assign(n, 0);
    tmax->assign(n, 0);
    for (size_t i = 0; i < n; i++) {
        const VPlan &vp = P.v[i];
        const int v = vp.vi;
        uint64_t hi = g->maxL[v], lo;
        if (g->overridden) {
            hi = 0;
            lo = ~0ull;
            for (uint32_t c = 0; c < g->K[v]; c++) {
                hi = std::max(hi, g->ov_layer[g->ov_layer_off[v] + c]);
                lo = std::min(lo, g->ov_layer[g->ov_layer_off[v] + c]);
            }
        } else {
            // the exact cost of single configurations: unsplit (F: no partial
            // sums, no replicas), and each dim k split p ways; every term of
            // these is bounded by the parts of maxL, so nothing overflows
            const pase_vertex_desc &d = g->V[v];
            const uint64_t F = g->flops[v], W = g->weight_n[v], p = g->p;
            lo = F;
            for (uint32_t k = 0; k < d.ndims; k++) {
                uint64_t c = (F + p - 1) / p;
                if ((d.reduce_mask >> k) & 1u) c += g->r * (p - 1) * g->keep_n[v];
                if (W && !((d.weight_mask >> k) & 1u)) c += g->r * (2 * W - 2 * W / p);
                // the halo of the split dim itself: the other input dims are unsplit
                if (g->halo && d.halo[k]) c += g->r * 2 * (uint64_t)d.halo[k] * g->halo_n[v][k];
                lo = std::min(lo, c);
            }
        }
        uint64_t rest = 0;
        for (int e : vp.edges) {
            uint64_t m = g->maxR[e];
            if (g->overridden) {
                m = 0;
                const uint64_t cnt = (uint64_t)g->K[g->E[e].src] * g->K[g->E[e].dst];
                for (uint64_t k = 0; k < cnt; k++) m = std::max(m, g->ov_edge[g->ov_edge_off[e] + k]);
            }
            if (!add_ok(rest, m, &rest)) return false;
        }
        for (const TermRef &t : vp.terms)
            if (!add_ok(rest, (*tmax)[t.j], &rest)) return false;
        if (!add_ok(hi, rest, &(*qmax)[i]) || !add_ok(lo, rest, &(*tmax)[i])) return false;
    }
    return true;
}

// Key type: fp64 when every key (cost * 2^bits + c) of every position stays
// within 2^53 so that double arithmetic on them is exact integer arithmetic;
// otherwise uint64 when it stays within 2^64; otherwise 128-bit keys, which
// hold cost * 2^bits + c exactly as long as every cost sum fits 64 bits (the
// costs and tables the C ABI reports are uint64); when a cost bound itself
// passes 64 bits, overflow.  A stored table entry T_j (in its reader's key
// space) is at most the reader's bound.  key_mode 1 / 2 force uint64 (when
// the keys fit) / 128-bit keys.
uint32_t choose_key_type(pase_graph_t g, pase_status *st) {
    *st = PASE_OK;
    std::vector<uint64_t> qmax, tmax;
    if (!cost_bounds(g, &qmax, &tmax)) { *st = PASE_ERR_OVERFLOW; return 0; }
    unsigned __int128 top = 0;
    for (size_t i = 0; i < qmax.size(); i++) {
        // largest key: qmax * 2^bits + (2^bits - 1) < (qmax + 1) * 2^bits
        const unsigned __int128 t = ((unsigned __int128)qmax[i] + 1) << g->plan.v[i].bits;
        top = std::max(top, t);
    }
    if (g->key_mode == 2) return 2;
    if (g->key_mode == 0 && top <= ((unsigned __int128)1 << 53)) return 0;
    if (top <= ((unsigned __int128)1 << 64)) return 1;
    return 2;
}

uint32_t key_bytes(pase_graph_t g) { return g->plan_wide ? 16u : 8u; }

}  // namespace pase

// ------------------------------------------------------------------ create / destroy
extern "C" pase_status pase_graph_create(const pase_vertex_desc *v, uint32_t nv,
                                         const pase_edge_desc *e, uint32_t ne,
                                         const pase_cost_params *params, pase_graph_t *out) {
    if (!v || !out || nv == 0 || (ne > 0 && !e)) return PASE_ERR_INVALID_ARGUMENT;
    if (nv > (1u << 20) || ne > (1u << 24)) return PASE_ERR_INVALID_ARGUMENT;
    for (uint32_t i = 0; i < nv; i++) {
        if (v[i].ndims < 1 || v[i].ndims > kMaxDims) return PASE_ERR_INVALID_ARGUMENT;
        for (uint32_t k = 0; k < v[i].ndims; k++)
            if (v[i].size[k] == 0) return PASE_ERR_INVALID_ARGUMENT;
        if (v[i].reduce_mask >> v[i].ndims) return PASE_ERR_INVALID_ARGUMENT;
        if (v[i].weight_mask >> v[i].ndims) return PASE_ERR_INVALID_ARGUMENT;
        if (v[i].input_mask >> v[i].ndims) return PASE_ERR_INVALID_ARGUMENT;
        for (uint32_t k = 0; k < kMaxDims; k++)
            if (v[i].halo[k] && (k >= v[i].ndims || !((v[i].input_mask >> k) & 1u) || v[i].halo[k] > (1u << 16)))
                return PASE_ERR_INVALID_ARGUMENT;
    }
    for (uint32_t k = 0; k < ne; k++) {
        const pase_edge_desc &d = e[k];
        if (d.src >= nv || d.dst >= nv || d.src == d.dst) return PASE_ERR_INVALID_ARGUMENT;
        if (d.rank > kMaxDims || d.elems == 0) return PASE_ERR_INVALID_ARGUMENT;
        for (uint32_t t = 0; t < d.rank; t++) {
            if (d.src_dim[t] < -1 || d.src_dim[t] >= (int32_t)v[d.src].ndims)
                return PASE_ERR_INVALID_ARGUMENT;
            if (d.dst_dim[t] < -1 || d.dst_dim[t] >= (int32_t)v[d.dst].ndims)
                return PASE_ERR_INVALID_ARGUMENT;
        }
    }
    auto *g = new pase_graph_s();
    g->V.assign(v, v + nv);
    if (ne) g->E.assign(e, e + ne);
    if (params) {
        g->r = params->comm_weight ? params->comm_weight : 8;
        if (params->seq_rule > 1) { delete g; return PASE_ERR_INVALID_ARGUMENT; }
        g->seq_rule = params->seq_rule;
    }
    g->nbr.assign(nv, {});
    for (const auto &d : g->E) {
        g->nbr[d.src].push_back((int)d.dst);
        g->nbr[d.dst].push_back((int)d.src);
    }
    for (auto &l : g->nbr) {
        std::sort(l.begin(), l.end());
        l.erase(std::unique(l.begin(), l.end()), l.end());
    }
    // weak connectivity (computation graphs are weakly connected, Sec. II)
    std::vector<char> seen(nv, 0);
    std::vector<int> stack{0};
    seen[0] = 1;
    size_t count = 1;
    while (!stack.empty()) {
        int x = stack.back();
        stack.pop_back();
        for (int y : g->nbr[x])
            if (!seen[y]) { seen[y] = 1; count++; stack.push_back(y); }
    }
    if (count != nv) { delete g; return PASE_ERR_NOT_CONNECTED; }
    *out = g;
    return PASE_OK;
}

extern "C" void pase_graph_destroy(pase_graph_t g) {
    if (!g) return;
    device_release(g);
    delete g;
}

extern "C" const char *pase_last_error(pase_graph_t g) { return g ? g->err.c_str() : ""; }

// ------------------------------------------------------------------ planning
namespace {

// Breadth-first traversal from vertex 0, neighbours in ascending id order:
// the sequence of the breadth-first recurrence (eq. 2).
std::vector<int> bfs_order(pase_graph_t g) {
    const size_t n = g->V.size();
    std::vector<int> order;
    order.reserve(n);
    std::vector<char> seen(n, 0);
    order.push_back(0);
    seen[0] = 1;
    for (size_t h = 0; h < order.size(); h++)
        for (int u : g->nbr[order[h]])      // ascending, deduplicated
            if (!seen[u]) { seen[u] = 1; order.push_back(u); }
    return order;
}

// GenerateSeq (Fig. 3): repeatedly sequence the unsequenced vertex with the
// smallest d-set (ties: lowest vertex id); every member of its d-set absorbs
// it.  rule 0 keeps a vertex out of its own d-set; rule 1 applies the printed
// update literally.  The d-set at selection (minus the vertex) is D(i)
// (Theorem 2).  Bitsets, one per vertex.  With a fixed `order` the same
// absorption runs along that order instead of the smallest-d-set choice: the
// d-set of a vertex then still holds the unsequenced neighbours of the
// sequenced component it would join, so at selection it is D(i) =
// N(X(i)) after i for that order (for a breadth-first order, D_B(i)).
void generate_seq(pase_graph_t g, std::vector<int> &seq, std::vector<std::vector<int>> &Dpos,
                  const std::vector<int> *order = nullptr) {
    const size_t n = g->V.size(), W = (n + 63) / 64;
    std::vector<uint64_t> d(n * W, 0);
    for (size_t v = 0; v < n; v++)
        for (int u : g->nbr[v]) d[v * W + u / 64] |= 1ull << (u % 64);
    // |u.d| is kept per vertex and recounted only when u.d changes
    auto count = [&](size_t u) {
        int sz = 0;
        for (size_t w = 0; w < W; w++) sz += __builtin_popcountll(d[u * W + w]);
        return sz;
    };
    std::vector<int> size(n);
    for (size_t u = 0; u < n; u++) size[u] = count(u);
    // vertices not sequenced yet, in no particular order: the pick is the
    // smallest (|u.d|, vertex id), so the scan order does not matter
    std::vector<int> left(n), where(n);
    std::iota(left.begin(), left.end(), 0);
    std::iota(where.begin(), where.end(), 0);
    seq.clear();
    Dpos.assign(n, {});
    for (size_t i = 0; i < n; i++) {
        size_t best = n;
        if (order) {
            best = (size_t)(*order)[i];
        } else {
            for (int u : left)
                if (best == n || size[u] < size[best] || (size[u] == size[best] && (size_t)u < best)) best = (size_t)u;
        }
        const size_t vi = best;
        // remove vi from the unsequenced set (swap with the last)
        const int at = where[vi], tail = left.back();
        left[at] = tail;
        where[tail] = at;
        left.pop_back();
        seq.push_back((int)vi);
        // D(i) = vi.d (ascending vertex id): the set bits of its row
        for (size_t w = 0; w < W; w++)
            for (uint64_t bits = d[vi * W + w]; bits; bits &= bits - 1) {
                const size_t u = w * 64 + (size_t)__builtin_ctzll(bits);
                if (u != vi) Dpos[i].push_back((int)u);
            }
        for (int v : Dpos[i]) {
            for (size_t w = 0; w < W; w++) d[(size_t)v * W + w] |= d[vi * W + w];
            d[(size_t)v * W + vi / 64] &= ~(1ull << (vi % 64));
            if (g->seq_rule == 0) d[(size_t)v * W + v / 64] &= ~(1ull << (v % 64));
            size[v] = count((size_t)v);
        }
    }
}

// column chunk widths of the row kernel (keys per lane and c, read as one
// scalar round trip of up to two s_load_dwordx16 plus a smaller load)
const uint32_t kTZ[] = {8, 12, 14, 16, 24, 28};

struct RowsChoice {
    bool ok = false;
    double cost = 0;
    int z = -1;
    std::vector<int> O, R;
    uint32_t TZ = 0, TM = 1, na = 0, parts = 1, nsplit = 1;
    uint64_t MO = 1, MR = 1;
};

// Estimated fill time (us) of one row-kernel vertex for a tile shape, with the
// best number of c parts per tile (waves of a workgroup) and c splits (across
// workgroups) -- or the forced ones.  The time is the larger of the throughput
// bound (the busiest SIMD's waves, each issuing a VALU op every 4 cycles) and
// the latency bound of a single wave: per value of c at least one memory round
// trip for the operands prefetched one c ahead (~450 cycles; column-less tiles
// keep 8 values of c in flight, ~360 cycles per c), or its own VALU work at
// about one op per 8 cycles.  Column-less tiles also stream their large
// lookups (stream_bytes: the multi-digit tables they read, each entry once;
// the one-digit row blocks stay in cache) at ~3.3 TB/s; when that stream binds,
// the estimates of several part counts tie, and the most parts win: more
// waves keep more loads in flight (measured on the Transformer's streaming
// fills: 287 us with one part, 244 us with two or four).  A c split adds a
// reduction launch (~10 us with its gap) and the partial keys' traffic; the
// column block is built at ~115 G elements/s.
struct TileTime {
    double us;
    uint32_t parts, nsplit;
};

TileTime tile_time(uint64_t MO, uint64_t MR, uint32_t Kz, uint32_t K, uint32_t na, uint32_t tz, uint32_t tm,
                   uint32_t force_parts, uint32_t force_splits, double stream_bytes) {
    const double clk = 2400.0;   // cycles per us
    const uint64_t nch = (Kz + tz - 1) / tz;
    const uint64_t tiles = MO * ((MR + 64 * tm - 1) / (64 * tm)) * nch;
    const uint64_t N = MO * MR * (uint64_t)Kz;
    const double prep_us = (double)MO * K * nch * tz / 1.15e5;
    TileTime best{1e300, 1, 1};
    for (uint32_t P = 1; P <= 4; P *= 2) {
        if (force_parts && P != force_parts) continue;
        for (uint32_t S = 1; S <= 64; S *= 2) {
            if (force_splits && S != 1) break;
            const uint32_t Sx = force_splits ? std::min(force_splits, K) : S;
            if (!force_splits && S > 1 && K < 8 * P * S) break;
            const double cw = std::ceil(std::ceil((double)K / Sx) / P);
            double wave_cyc, lat_cyc, bw_us = 0;
            if (tz >= 8) {
                // VALU slots per c: two per cell, the row-term adds, and (measured)
                // a few for wide chunks (> 16 keys: no scalar-load overlap) and
                // for two rows per lane (more VGPRs, fewer waves).  Every row-term
                // load is a wave-wide vector load that keeps the CU's texture
                // address unit ~16 cycles busy; shared by four SIMDs, that costs
                // ~15 VALU slots per load per wave when all SIMDs are busy; the
                // two overlap imperfectly (fitted: the smaller adds a quarter).
                const double valu = 2.0 * tz * tm + tm * (na > 0 ? na - 1.0 : 0.0) + 1.0 + (tz > 16 ? 2.0 : 0.0) +
                                    (tm == 2 ? 2.0 : 0.0);
                const double ta = 14.7 * na * tm;
                double per_c = std::max(valu, ta) + 0.25 * std::min(valu, ta);
                // a column block larger than the L2s is read from HBM: a scalar
                // round trip then takes ~2000 cycles, ~60 slots per wave with
                // eight waves per SIMD -- hidden behind one c of work when the
                // loads of c + 1 are in flight (up to 16 keys), exposed when not
                if ((double)MO * K * nch * tz * 8 > 16e6) per_c = tz > 16 ? per_c + 62.0 : std::max(per_c, 62.0);
                const double tail = tz * tm * (P > 1 ? 8.0 : 6.0);
                wave_cyc = 4.0 * (cw * per_c + tail);
                lat_cyc = cw * std::max(8.0 * per_c, 450.0) + 8.0 * tail;
            } else {
                wave_cyc = 4.0 * cw * (2.0 * tm + tm * (na > 0 ? na - 1.0 : 0.0) + 1.0);
                lat_cyc = 360.0 * cw;
                bw_us = stream_bytes / 3.3e6;
            }
            // the busiest SIMD: the average share plus, on average, half a wave
            const double W = (double)tiles * P * Sx;
            const double t_tp = (W / 1024.0 + 0.5) * wave_cyc / clk;
            double us = std::max(std::max(t_tp, lat_cyc / clk), bw_us) + prep_us;
            if (Sx > 1) us += 10.0 + (double)N * Sx * 16 / 5e6;
            // parts ascend: a column-less tie goes to the later, larger count
            const bool tie_more_parts = tz < 8 && Sx == 1 && best.nsplit == 1 && us <= best.us * (1.0 + 1e-9);
            if (us < best.us || tie_more_parts) best = {us, P, Sx};
        }
    }
    return best;
}

// Vertices of one graph often share a shape (the layers of a stack): the tile
// model is evaluated once per distinct argument tuple.
TileTime tile_time_cached(uint64_t MO, uint64_t MR, uint32_t Kz, uint32_t K, uint32_t na, uint32_t tz, uint32_t tm,
                          uint32_t force_parts, uint32_t force_splits, double stream_bytes) {
    struct Key {
        uint64_t MO, MR;
        uint32_t Kz, K, na, tz, tm, parts, splits;
        double sb;
        bool operator==(const Key &o) const {
            return MO == o.MO && MR == o.MR && Kz == o.Kz && K == o.K && na == o.na && tz == o.tz && tm == o.tm &&
                   parts == o.parts && splits == o.splits && sb == o.sb;
        }
    };
    struct Hash {
        size_t operator()(const Key &k) const {
            uint64_t h = k.MO * 0x9E3779B97F4A7C15ull ^ (k.MR + 0x632BE59BD9B4E019ull) ^ (uint64_t)k.sb;
            for (uint32_t x : {k.Kz, k.K, k.na, k.tz, k.tm, k.parts, k.splits}) h = (h ^ x) * 0x100000001B3ull;
            return (size_t)h;
        }
    };
    thread_local std::unordered_map<Key, TileTime, Hash> memo;
    const Key key{MO, MR, Kz, K, na, tz, tm, force_parts, force_splits, stream_bytes};
    auto it = memo.find(key);
    if (it != memo.end()) return it->second;
    if (memo.size() > 65536) memo.clear();
    const TileTime t = tile_time(MO, MR, Kz, K, na, tz, tm, force_parts, force_splits, stream_bytes);
    memo.emplace(key, t);
    return t;
}

}  // namespace

// Fused minima.  A row-kernel vertex i2 without a column digit whose only
// lookup is the table of i1 -- a row-kernel vertex whose column digit is v_i2,
// with no outer digits, the same row digits and neither of them split over c
// -- streams all of T_i1 once to take, per row, a minimum over c = z.  i1's fill
// forms those keys itself in its epilogue instead (T_i1 has no other reader),
// so T_i1 is neither written to nor read back from HBM, and i2 keeps a
// one-split reduction of the combined keys.  i2's prep blocks hold static
// costs only (its one lookup is read in the kernel), so they are built in
// i1's prep launch, before i1's fill.  Both run on one lane.
static void fuse_minima(pase_graph_t g, Plan &P) {
    (void)g;
    const int n = (int)P.v.size();
    for (int i2 = 0; i2 < n; i2++) {
        VPlan &b = P.v[i2];
        if (b.kernel != kRows || b.z >= 0 || b.nsplit != 1 || b.terms.size() != 1 || b.terms[0].dig.size() < 2)
            continue;
        const int i1 = b.terms[0].j;
        VPlan &a = P.v[i1];
        if (a.kernel != kRows || a.z != b.vi || !a.O.empty() || a.R != b.R || a.nsplit != 1 || a.consumer != i2 ||
            a.lane != b.lane || a.fuse_into >= 0 || a.fused_from >= 0)
            continue;
        a.fuse_into = i2;
        b.fused_from = i1;
        P.fused++;
    }
}

// Hoisted preps (level layout: one stream, slots = levels).  A vertex's prep builds its key-space blocks
// from static costs and from the tables of the lookups that enter blocks (the
// column block's and the one-digit row blocks'; multi-digit lookups on row
// digits are read by the fill itself).  When the last of those tables is
// filled two or more slots before the vertex's own, and the blocks are large
// (PASE_OPT_HOIST_ELEMS, by default 2^20 elements: ~10 us or more of HBM
// writes), the prep runs on a side stream instead of in the vertex's slot,
// started right after that slot, on a grid of one workgroup per CU: it then
// takes several times longer but leaves most of the GPU to the launches of
// the slots in between (a full-size prep grid beside them slows them down
// more than it saves).
static void hoist_preps(pase_graph_t g, Plan &P, bool lanes) {
    for (auto &vp : P.v) {
        if ((vp.kernel != kRows && vp.kernel != kGeneric) || vp.fused_from >= 0 || vp.fuse_into >= 0) continue;
        uint64_t elems = 0;
        int ready = -1;
        int lane = -1;            // lane of the tables the blocks read (-2: more than one)
        auto note = [&](int j) {
            ready = std::max(ready, P.v[j].slot);
            lane = lane == -1 || lane == P.v[j].lane ? P.v[j].lane : -2;
        };
        if (vp.kernel == kRows) {
            elems = vp.MO * vp.K * vp.ldz;
            for (int u : vp.R) elems += (uint64_t)vp.K * g->K[u];
            std::vector<int> OZ = vp.O;
            if (vp.z >= 0) OZ.push_back(vp.z);
            for (const auto &t : vp.terms) {
                bool all = true;
                for (int u : t.dig) all &= std::find(OZ.begin(), OZ.end(), u) != OZ.end();
                const bool row1 = t.dig.size() == 1 && std::count(vp.R.begin(), vp.R.end(), t.dig[0]);
                if (all || row1) note(t.j);
            }
        } else {
            elems = vp.K;
            for (int u : vp.D) elems += (uint64_t)vp.K * g->K[u];
            for (const auto &t : vp.terms)
                if (t.dig.size() <= 1) note(t.j);
        }
        // with lanes, the prep runs at the end of the group (slot `ready`, at
        // least 0) of the lane whose tables it reads (the vertex's own when it
        // reads none): stream order puts it after those fills, and the
        // vertex's group waits for that lane up to that slot anyway -- or
        // shares its stream -- so the prep precedes the fill
        if (lanes) {
            if (lane == -2) continue;
            ready = std::max(ready, 0);
        }
        if (g->hoist_elems && elems >= g->hoist_elems && ready + 2 <= vp.slot) {
            vp.prep_after = ready;
            vp.prep_lane = lanes && lane >= 0 ? lane : vp.lane;
            P.hoisted++;
        }
    }
}

// Bulk lane schedule.  Row-kernel vertices planned to take at least bulk_us
// (the large fills, which keep the whole GPU busy on their own) run on lane 1
// (a stream of its own), and so does every vertex that reads a table of lane 1
// (it has to wait for that fill anyway); every other vertex -- one whose
// producers are all small -- runs on lane 0 (the caller's stream), level by
// level, at the highest wave priority.  A level group of lane 0 then never
// waits for a large fill, so a chain of small dependent vertices runs beside
// the large fills instead of after them.  Producers precede their reader in
// the sequence, so one pass suffices.
static void assign_bulk_lanes(Plan &P, double bulk_us) {
    for (auto &vp : P.v) {
        bool bulk = vp.kernel == kRows && vp.est_us >= bulk_us;
        for (const auto &t : vp.terms) bulk |= P.v[t.j].lane == 1;
        vp.lane = bulk ? 1 : 0;
    }
}

// Split chains schedule.  The first kSplitBatchedLevels levels -- the leaves,
// where the largest fills and most small vertices are -- run level by level
// on lane 1, batched as in the level schedule.  After them, a row-kernel
// vertex planned at bulk_us or more, and every vertex reading a table such a
// vertex (or one of its readers) fills after the batched levels, runs on lane
// 1 too; the remaining small vertices run on lane 0.  A lane-0 group waits
// once for the batched levels whose tables it reads and then runs beside lane
// 1, so a chain of small vertices and a chain of larger fills no longer wait
// for each other level by level.
static void assign_split_lanes(Plan &P, double bulk_us) {
    for (auto &vp : P.v) {
        bool one = vp.level < kSplitBatchedLevels || (vp.kernel == kRows && vp.est_us >= bulk_us);
        for (const auto &t : vp.terms) one |= P.v[t.j].lane == 1 && P.v[t.j].level >= kSplitBatchedLevels;
        vp.lane = one ? 1 : 0;
    }
}

static double ms_since(std::chrono::steady_clock::time_point t0) {
    return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
}

static pase_status build_plan(pase_graph_t g) {
    const auto t0 = std::chrono::steady_clock::now();
    const int n = (int)g->V.size();
    Plan &P = g->plan;
    P = Plan();
    std::vector<std::vector<int>> Dpos;
    if (g->order_mode == 1) {
        const std::vector<int> order = bfs_order(g);
        generate_seq(g, P.seq, Dpos, &order);
    } else {
        generate_seq(g, P.seq, Dpos);
    }
    P.pos.assign(n, 0);
    for (int i = 0; i < n; i++) P.pos[P.seq[i]] = i;
    P.v.assign(n, VPlan());

    // edges of each vertex, in edge order
    std::vector<std::vector<int>> incident(n);
    for (size_t k = 0; k < g->E.size(); k++) {
        incident[g->E[k].src].push_back((int)k);
        incident[g->E[k].dst].push_back((int)k);
    }
    // components of the graph induced on positions < i, grown one position at
    // a time (union-find over vertex ids); each set remembers its last position
    std::vector<int> uf(n), last(n, -1), seen(n, -1);
    std::iota(uf.begin(), uf.end(), 0);
    auto find = [&](int x) {
        while (uf[x] != x) x = uf[x] = uf[uf[x]];
        return x;
    };
    for (int i = 0; i < n; i++) {
        VPlan &vp = P.v[i];
        vp.vi = P.seq[i];
        vp.K = g->K[vp.vi];
        vp.bits = bits_for(vp.K);
        vp.D = Dpos[i];
        std::sort(vp.D.begin(), vp.D.end());
        if (vp.D.size() > (size_t)kMaxDep)
            return fail(g, PASE_ERR_TOO_LARGE, "dependent set larger than PASE_MAX_DEP");
        P.max_dep = std::max<uint32_t>(P.max_dep, (uint32_t)vp.D.size());
        vp.N = 1;
        for (int w : vp.D)
            if (!mul_ok(vp.N, g->K[w], &vp.N) || vp.N > kMaxTableEntries)
                return fail(g, PASE_ERR_TOO_LARGE, "a DP table exceeds 2^31 entries");
        // S(i): the components of V<i that v_i touches, each represented by its
        // last position j (X(i) - {v_i} is their union)
        for (int s : g->nbr[vp.vi]) {
            if (P.pos[s] >= i) continue;
            const int rt = find(s);
            if (seen[rt] == i) continue;
            seen[rt] = i;
            const int jmax = last[rt];
            TermRef t;
            t.j = jmax;
            bool has_vi = false;
            for (int u : P.v[jmax].D) {
                if (u == vp.vi) { has_vi = true; continue; }
                if (!std::binary_search(vp.D.begin(), vp.D.end(), u))
                    return fail(g, PASE_ERR_INTERNAL, "D(j) not within D(i) + v_i");
                t.dig.push_back(u);
            }
            if (!has_vi) return fail(g, PASE_ERR_INTERNAL, "v_i missing from D(j)");
            if (P.v[jmax].consumer != -1) return fail(g, PASE_ERR_INTERNAL, "table read twice");
            P.v[jmax].consumer = i;
            vp.terms.push_back(t);
        }
        // v_i joins the components it touches and is their last position
        last[vp.vi] = i;
        for (int s : g->nbr[vp.vi])
            if (P.pos[s] < i) {
                const int a = find(s), b = find(vp.vi);
                if (a != b) uf[a] = b;
            }
        last[find(vp.vi)] = i;
        for (int k : incident[vp.vi]) {
            const auto &d = g->E[k];
            const int other = (int)d.src == vp.vi ? (int)d.dst : (int)d.src;
            if (P.pos[other] > i) vp.edges.push_back(k);
        }
        P.cells += vp.N * vp.K;
        P.entries += vp.N;
    }
    for (int i = 0; i + 1 < n; i++) {
        if (P.v[i].consumer < 0) return fail(g, PASE_ERR_INTERNAL, "table never read");
        P.v[i].out_shift = P.v[P.v[i].consumer].bits;
    }
    g->stats.seq_ms = ms_since(t0);
    const auto t1 = std::chrono::steady_clock::now();
    // dependency level: vertices of one level read no table of each other
    for (int i = 0; i < n; i++) {
        P.v[i].level = 0;
        for (const auto &t : P.v[i].terms) P.v[i].level = std::max(P.v[i].level, P.v[t.j].level + 1);
    }

    // ---- kernel choice and T_i layout
    // threads of the generic and direct fills walk the table in layout order:
    // follow the memory order of the largest lookup that spans several digits
    // so that its reads coalesce
    auto gather_layout = [&](const VPlan &vp) {
        int big = -1;
        for (size_t t = 0; t < vp.terms.size(); t++)
            if (vp.terms[t].dig.size() >= 2 && (big < 0 || P.v[vp.terms[t].j].N > P.v[vp.terms[big].j].N))
                big = (int)t;
        if (big < 0) return vp.D;
        const VPlan &pj = P.v[vp.terms[big].j];
        std::vector<int> order;
        for (int u : pj.layout)
            if (u != vp.vi) order.push_back(u);   // slowest first in T_j
        for (int u : vp.D)
            if (std::find(order.begin(), order.end(), u) == order.end()) order.insert(order.begin(), u);
        return order;
    };
    // the direct fill pays where it removes launches: for a whole level (the
    // vertices of one launch group), or any vertex when each has its own slot
    int maxlev = 0;
    for (int i = 0; i < n; i++) maxlev = std::max(maxlev, P.v[i].level);
    std::vector<char> level_small((size_t)maxlev + 1, 1);
    for (int i = 0; i < n; i++)
        if (P.v[i].N * P.v[i].K > g->direct_cells) level_small[P.v[i].level] = 0;
    // plan_one(i, ftz, ftm, no_split): kernel, tile and layout of position i;
    // ftz/ftm (0 = free) force the row kernel's columns and rows per lane for
    // this vertex and rule out the column-less form; no_split rules out a c
    // split
    // 128-bit keys: every vertex on prep + the generic kernel
    const int kernel_mode = g->plan_wide ? 1 : g->kernel_mode;
    auto plan_one = [&](int i, uint32_t ftz, uint32_t ftm, bool no_split) {
        VPlan &vp = P.v[i];
        const uint32_t tile_cols = ftz ? ftz : g->tile_cols, tile_rows = ftm ? ftm : g->tile_rows;
        // small vertices: the direct fill (one launch, no prep blocks), whose
        // time is a launch plus the gather of every term of every cell
        if (!ftz && g->direct_cells && kernel_mode == 0 && vp.N * vp.K <= g->direct_cells && (g->schedule == kSchedSeq || level_small[vp.level])) {
            vp.kernel = kDirect;
            vp.est_us = 4.0 + (double)vp.N * vp.K * (1.0 + vp.edges.size() + vp.terms.size()) / 4e5;
            vp.layout = gather_layout(vp);
            vp.nsplit = 1;
            vp.cper = vp.K;
            vp.stride.assign(vp.layout.size(), 1);
            for (int k = (int)vp.layout.size() - 2; k >= 0; k--)
                vp.stride[k] = vp.stride[k + 1] * g->K[vp.layout[k + 1]];
            return;
        }
        RowsChoice best;
        // candidates: every digit of D(i) as the column digit z, and -- only
        // when none of those fits -- no column at all (z = -1: every digit is
        // a row digit, each lane streams its own entry's terms over c; for a
        // lookup that covers all of D(i) this reads T_j once, coalesced)
        std::vector<int> zs;
        if (kernel_mode == 0 && vp.D.size() >= 2) zs = vp.D;
        if (kernel_mode == 0 && !vp.D.empty() && !ftz) zs.push_back(-1);
        for (int z : zs) {
            if (z < 0 && best.ok) break;
            {
                RowsChoice rc;
                rc.z = z;
                std::vector<int> O;
                for (const auto &t : vp.terms)
                    if (z >= 0 && t.dig.size() >= 2 && std::count(t.dig.begin(), t.dig.end(), z))
                        for (int u : t.dig)
                            if (u != z) O.push_back(u);
                std::sort(O.begin(), O.end());
                O.erase(std::unique(O.begin(), O.end()), O.end());
                for (int u : vp.D)
                    if (u != z && !std::binary_search(O.begin(), O.end(), u)) rc.R.push_back(u);
                rc.O = O;
                for (int u : rc.O) rc.MO *= g->K[u];
                for (int u : rc.R) rc.MR *= g->K[u];
                if (rc.MR < (z < 0 ? 256u : 16u)) continue;
                uint32_t na = 0;
                for (int u : rc.R) {
                    bool used = false;
                    for (int e : vp.edges) {
                        int other = (int)g->E[e].src == vp.vi ? (int)g->E[e].dst : (int)g->E[e].src;
                        used |= other == u;
                    }
                    for (const auto &t : vp.terms) used |= t.dig.size() == 1 && t.dig[0] == u;
                    na += used;
                }
                bool small = true;   // row terms are read with 32-bit buffer offsets
                double stream_bytes = 0;
                for (const auto &t : vp.terms) {
                    if (t.dig.size() < 2) continue;
                    bool touches = false;
                    for (int u : t.dig) touches |= std::binary_search(rc.R.begin(), rc.R.end(), u);
                    na += touches;
                    if (touches && P.v[t.j].N * 8 >= (1ull << 31)) small = false;
                    if (touches) stream_bytes += 8.0 * (double)std::min<uint64_t>(P.v[t.j].N, vp.N * vp.K);
                }
                if (na > (uint32_t)kMaxATerms || !small) continue;
                rc.na = na;
                const uint32_t Kz = z >= 0 ? g->K[z] : 1;
                static const uint32_t kNoColumn[] = {1};
                for (uint32_t tz : z >= 0 ? std::vector<uint32_t>(std::begin(kTZ), std::end(kTZ))
                                          : std::vector<uint32_t>(std::begin(kNoColumn), std::end(kNoColumn))) {
                    if (z >= 0 && tile_cols && tz != tile_cols) continue;
                    uint64_t nch = (Kz + tz - 1) / tz;
                    if (rc.MO * vp.K * nch * tz > kMaxTableEntries) continue;
                    for (uint32_t tm = 1; tm <= 2; tm++) {
                        if (tile_rows && tm != tile_rows) continue;
                        // more than 32 accumulators per lane cost waves (VGPRs)
                        if (!tile_rows && !tile_cols && tz * tm > 32) continue;
                        const TileTime tt = tile_time_cached(rc.MO, rc.MR, Kz, vp.K, na, tz, tm, g->tile_parts,
                                                             no_split ? 1u : g->c_splits, stream_bytes);
                        if (!rc.ok || tt.us < rc.cost) {
                            rc.ok = true;
                            rc.cost = tt.us;
                            rc.TZ = tz;
                            rc.TM = tm;
                            rc.parts = tt.parts;
                            rc.nsplit = tt.nsplit;
                        }
                    }
                }
                if (rc.ok && (!best.ok || rc.cost < best.cost)) best = rc;
            }
        }
        if (best.ok) {
            vp.kernel = kRows;
            vp.z = best.z;
            vp.O = best.O;
            vp.R = best.R;
            vp.MO = best.MO;
            vp.MR = best.MR;
            vp.TZ = best.TZ;
            vp.TM = best.TM;
            vp.na = best.na;
            vp.nchunks = ((vp.z >= 0 ? g->K[vp.z] : 1) + vp.TZ - 1) / vp.TZ;
            vp.ldz = vp.nchunks * vp.TZ;
            vp.layout.clear();
            if (vp.z >= 0) vp.layout.push_back(vp.z);
            vp.layout.insert(vp.layout.end(), vp.O.begin(), vp.O.end());
            vp.layout.insert(vp.layout.end(), vp.R.begin(), vp.R.end());
            vp.parts = best.parts;
            vp.est_us = best.cost;
            const uint64_t ns = best.nsplit;
            vp.cper = (uint32_t)((vp.K + ns - 1) / ns);
            vp.nsplit = (vp.K + vp.cper - 1) / vp.cper;
        } else {
            vp.kernel = kGeneric;
            // gather-bound: ~1e11 cell updates/s, plus a launch's worth of latency
            vp.est_us = 5.0 + (double)vp.N * vp.K / 1e5;
            vp.layout = gather_layout(vp);
            vp.nsplit = 1;
            vp.cper = vp.K;
        }
        vp.stride.assign(vp.layout.size(), 1);
        for (int k = (int)vp.layout.size() - 2; k >= 0; k--)
            vp.stride[k] = vp.stride[k + 1] * g->K[vp.layout[k + 1]];
    };
    for (int i = 0; i < n; i++) plan_one(i, 0, 0, false);
    // One launch per level and kernel variant: a small column-form row vertex
    // of a level is re-planned with the tile shape of the level's largest one
    // when its fill then stays under half of that vertex's, so that the two
    // share a launch (the small one's workgroups come first and finish inside
    // the large one's) instead of adding a latency-bound launch of its own.
    // When the largest one is not split over c, the small one is not either:
    // its latency is hidden in the shared launch anyway, and a split would
    // only add the level's reduction launch.
    // Level schedule only: the bulk lane splits a level over two streams.
    if ((g->schedule == kSchedLevel || g->schedule == kSchedSplit) && !g->tile_cols && !g->tile_rows &&
        kernel_mode == 0) {
        std::vector<int> dom((size_t)maxlev + 1, -1);
        for (int i = 0; i < n; i++) {
            const VPlan &vp = P.v[i];
            if (vp.kernel != kRows || vp.z < 0) continue;
            int &d = dom[vp.level];
            if (d < 0 || vp.est_us > P.v[d].est_us) d = i;
        }
        for (int i = 0; i < n; i++) {
            const int d = dom[P.v[i].level];
            if (d < 0 || d == i || P.v[i].kernel != kRows || P.v[i].z < 0) continue;
            // (split chains: only the batched levels share launches level-wide)
            if (g->schedule == kSchedSplit && P.v[i].level >= kSplitBatchedLevels) continue;
            const VPlan &dv = P.v[d];
            const bool unsplit = dv.nsplit == 1 && !g->c_splits;
            if (P.v[i].TZ == dv.TZ && P.v[i].TM == dv.TM && (!unsplit || P.v[i].nsplit == 1)) continue;
            const VPlan saved = P.v[i];
            plan_one(i, dv.TZ, dv.TM, unsplit);
            const VPlan &nv = P.v[i];
            const bool ok = nv.kernel == kRows && nv.z >= 0 && nv.TZ == dv.TZ && nv.TM == dv.TM &&
                            nv.na <= dv.na && nv.est_us <= 0.5 * dv.est_us;
            if (!ok) P.v[i] = saved;
        }
    }
    for (const auto &vp : P.v) {
        if (vp.kernel != kRows) continue;
        P.rows_vertices++;
        P.rows_cells += vp.N * vp.K;
        if (vp.z < 0) P.stream_cells += vp.N * vp.K;
    }
    for (auto &vp : P.v) vp.lane = 0;
    if (g->schedule == kSchedBulk) assign_bulk_lanes(P, (double)g->bulk_us);
    if (g->schedule == kSchedSplit) assign_split_lanes(P, (double)g->bulk_us);
    if (g->fuse_min && kernel_mode == 0) fuse_minima(g, P);
    g->stats.plan_ms = ms_since(t1);
    return PASE_OK;
}

// Device memory layout: constant region (configurations, vertex/edge
// descriptors, layer costs, caller-given edge matrices, prep contributions,
// back-substitution descriptors), outputs, the table arenas and scratch.
// Cost tables T_i live from their fill to their single reader (or to the end
// when tables are kept or i is last) and share memory by interval packing;
// argmin tables A_i all live until back-substitution.
enum LayoutMode { kLayoutResident = 0, kLayoutSeq = 1, kLayoutLevel = 2 };
static pase_status layout_memory_mode(pase_graph_t g, LayoutMode mode);

// The bulk lane schedule runs vertices of two streams concurrently and needs
// every table and scratch buffer resident at once; when that exceeds the
// budget, or for the level schedule, tables share memory by lifetimes over
// levels; when even that does not fit, one vertex at a time.
static pase_status layout_memory(pase_graph_t g) {
    const auto t0 = std::chrono::steady_clock::now();
    pase_status st = PASE_ERR_TOO_LARGE;
    if (g->schedule == kSchedBulk || g->schedule == kSchedSplit) st = layout_memory_mode(g, kLayoutResident);
    if (st != PASE_OK && g->schedule != kSchedSeq) st = layout_memory_mode(g, kLayoutLevel);
    if (st != PASE_OK) st = layout_memory_mode(g, kLayoutSeq);
    g->stats.plan_ms += ms_since(t0);
    g->stats.host_plan_ms = g->stats.seq_ms + g->stats.plan_ms;
    return st;
}

static pase_status layout_memory_mode(pase_graph_t g, LayoutMode mode) {
    Plan &P = g->plan;
    // resident: vertices may run in any order the dependencies allow, so
    // every vertex has scratch of its own and no table memory is reused
    const bool resident = mode == kLayoutResident, by_level = mode != kLayoutSeq;
    const uint64_t kb = key_bytes(g);   // bytes per table value and block key
    P.by_level = by_level;
    P.resident = resident;
    P.nslots = 0;
    for (auto &vp : P.v) {
        vp.slot = by_level ? vp.level : (int)(&vp - &P.v[0]);
        P.nslots = std::max(P.nslots, vp.slot + 1);
        vp.prep_after = -2;
    }
    P.hoisted = 0;
    if (mode == kLayoutLevel) hoist_preps(g, P, false);
    if (resident && (g->schedule == kSchedBulk || g->schedule == kSchedSplit)) hoist_preps(g, P, true);
    const int n = (int)P.v.size();
    const uint64_t A = 256;
    uint64_t off = 0;
    P.off_ex = off;
    for (const auto &rows : g->ex_rows) off += rows.size();   // one row set per dimension count
    off = align_up(off, A);
    P.off_vert = off;
    off = align_up(off + g->V.size() * sizeof(DevVertex), A);
    P.off_edge = off;
    off = align_up(off + std::max<size_t>(1, g->E.size()) * sizeof(DevEdge), A);
    P.off_L = off;
    uint64_t sumK = 0;
    for (uint32_t k : g->K) sumK += k;
    off = align_up(off + sumK * 8, A);
    P.off_lsum = off;
    off = align_up(off + sumK, A);
    P.sig_count = 0;
    for (const auto &d : g->E) P.sig_count += (uint64_t)g->K[d.src] + g->K[d.dst];
    P.off_sig = off;
    off = align_up(off + P.sig_count * 8, A);
    P.off_ovedge = off;
    if (g->overridden) off = align_up(off + g->ov_edge.size() * 8, A);
    // contributions: count per vertex (layer + edges + lookups is an upper bound)
    uint64_t ncontrib = 0;
    for (const auto &vp : P.v) ncontrib += 1 + vp.edges.size() + vp.terms.size();
    P.contrib_count = ncontrib;
    P.off_contrib = off;
    off = align_up(off + ncontrib * sizeof(Contrib), A);
    P.off_bt = off;
    off = align_up(off + n * sizeof(BacktrackDesc), A);
    P.off_desc = off;
    off = align_up(off + n * (sizeof(PrepArgs) + sizeof(RowsArgs) + sizeof(GenericArgs) + sizeof(ReduceArgs) +
                              sizeof(DirectArgs)), A);
    P.off_batch = off;
    off = align_up(off + 3 * (uint64_t)n * sizeof(BatchEntry), A);
    // one zero key: the row term that pads a row-kernel vertex up to the
    // row-term count of the launch it shares (uploaded zeroed with the rest)
    P.off_zero = off;
    off = align_up(off + 8, A);
    P.off_cfg = off;
    off = align_up(off + g->V.size() * 4, A);
    P.off_out = off;
    off = align_up(off + sizeof(SearchOut), A);
    // volume transfer model: the edge matrices are computed on the device, so
    // they sit past the uploaded constant region
    P.off_vmat = off;
    if (g->volume && !g->overridden) off = align_up(off + g->mat_total * 8, A);

    // T arena: interval packing over launch slots -- a table is written in the
    // slot of its vertex and last read in the slot of its reader
    struct Iv { int i, s, e; uint64_t size; };
    std::vector<Iv> iv;
    for (int i = 0; i < n; i++) {
        int end = (resident || g->keep_tables || i == n - 1) ? P.nslots : P.v[P.v[i].consumer].slot;
        iv.push_back({i, P.v[i].slot, end, align_up(P.v[i].N * kb, A)});
    }
    std::vector<int> order(n);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return iv[a].size > iv[b].size; });
    // placed tables in ascending offset order: the first gap that fits among
    // those whose lifetimes overlap is found in one pass
    std::vector<int> placed;
    placed.reserve(n);
    uint64_t tbytes = 0;
    for (int k : order) {
        uint64_t cand = 0;
        for (int q : placed) {
            if (!(iv[q].s <= iv[k].e && iv[k].s <= iv[q].e)) continue;
            const uint64_t b0 = P.v[iv[q].i].T_off;
            if (cand + iv[k].size <= b0) break;
            cand = std::max(cand, b0 + iv[q].size);
        }
        P.v[iv[k].i].T_off = cand;
        tbytes = std::max(tbytes, cand + iv[k].size);
        auto at = std::upper_bound(placed.begin(), placed.end(), cand,
                                   [&](uint64_t x, int q) { return x < P.v[iv[q].i].T_off; });
        placed.insert(at, k);
    }
    P.T_bytes = tbytes;
    P.off_T = off;
    off = align_up(off + tbytes, A);
    uint64_t abytes = 0;
    for (auto &vp : P.v) { vp.A_off = abytes; abytes += align_up(vp.N * 2, A); }
    P.A_bytes = abytes;
    P.off_A = off;
    off = align_up(off + abytes, A);
    // block and split scratch: vertices of one slot get disjoint pieces; slots reuse it
    std::vector<uint64_t> bsum(P.nslots, 0), psum(P.nslots, 0);
    uint64_t bmax = 0, pmax = 0;
    std::vector<VPlan *> hoisted;
    for (auto &vp : P.v) {
        uint64_t e = 0, pb = 0;
        if (vp.kernel == kRows) {
            e += align_up(vp.MO * vp.K * vp.ldz, 32);
            for (int u : vp.R) e += align_up((uint64_t)vp.K * g->K[u], 32);
            if (vp.nsplit > 1) pb = align_up((uint64_t)vp.nsplit * vp.N * kb, A);
        } else if (vp.kernel == kGeneric) {
            e += align_up(vp.K, 32);
            for (int u : vp.D) e += align_up((uint64_t)vp.K * g->K[u], 32);
        }   // the direct fill needs no prep blocks and no split scratch
        vp.block_elems = e;
        // (the resident layout keeps every vertex's scratch: one slot for all;
        // a fused minimum's blocks are built and read in its producer's slot)
        const int sl = resident ? 0 : vp.fused_from >= 0 ? P.v[vp.fused_from].slot : vp.slot;
        vp.partial_off = psum[sl];
        psum[sl] += pb;
        pmax = std::max(pmax, psum[sl]);
        if (vp.prep_after >= -1) {   // hoisted: blocks live from an earlier slot on
            hoisted.push_back(&vp);
            continue;
        }
        vp.block_off = bsum[sl];
        bsum[sl] += align_up(e * kb, A);
        bmax = std::max(bmax, bsum[sl]);
    }
    // hoisted blocks: after every slot's scratch, one piece each
    for (VPlan *vp : hoisted) {
        vp->block_off = bmax;
        bmax += align_up(vp->block_elems * kb, A);
    }
    P.block_bytes = bmax;
    P.off_block = off;
    off = align_up(off + P.block_bytes, A);
    P.partial_bytes = pmax;
    P.off_partial = off;
    off = align_up(off + P.partial_bytes, A);
    // keys of the fused minima: written in the producer's slot, read in the
    // reader's, so not shared with any other scratch
    P.fused_bytes = 0;
    for (auto &vp : P.v)
        if (vp.fused_from >= 0) {
            vp.fkeys_off = P.fused_bytes;
            P.fused_bytes += align_up(vp.N * kb, A);
        }
    P.off_fused = off;
    off = align_up(off + P.fused_bytes, A);
    P.total = off;
    if (P.total > g->mem_budget)
        return fail(g, PASE_ERR_TOO_LARGE, "device memory need exceeds the memory budget");
    return PASE_OK;
}

// Plan (or, with replan, re-plan from the vertex order on) the search: the
// key type that the plans and the current costs need (R10), then the memory
// layout.  A change to or from 128-bit keys re-plans every vertex (such plans
// run on the generic kernel).  OVERFLOW when a cost bound of the recurrence
// passes 64 bits.
static pase_status plan_search(pase_graph_t g, bool replan) {
    pase_status st;
    if (replan && (st = build_plan(g)) != PASE_OK) return st;
    const uint32_t kt = choose_key_type(g, &st);
    if (st != PASE_OK) return fail(g, st, "a cost bound of the recurrence exceeds 64 bits");
    if ((kt == 2) != g->plan_wide) {
        g->plan_wide = kt == 2;
        if ((st = build_plan(g)) != PASE_OK) return st;
    }
    g->plan_key_type = kt;
    return layout_memory(g);
}

extern "C" pase_status pase_enumerate_configs(pase_graph_t g, uint32_t p) {
    if (!g) return PASE_ERR_INVALID_ARGUMENT;
    const bool factors = g->config_set == 1;
    if (factors && (p == 0 || p > 255))
        return fail(g, PASE_ERR_INVALID_ARGUMENT, "p must be in 1..255 with every integer split");
    if (!factors && (p == 0 || (p & (p - 1)) || p > (1u << 16)))
        return fail(g, PASE_ERR_INVALID_ARGUMENT, "p must be a power of two <= 65536");
    g->enumerated = g->planned = g->searched = g->overridden = false;
    g->ov_layer.clear(); g->ov_edge.clear();
    g->p = p;
    g->factors = factors;
    g->volume = g->transfer_opt == 1;
    g->mat_off.assign(g->E.size(), 0);
    g->mat_total = 0;
    g->mat_row0.assign(g->E.size(), 0);
    g->mat_rows = 0;
    if (g->volume) {
        // the device's volume arithmetic needs Q = prod_t s_u(t) * s_v(t) < 2^32:
        // with distinct mapped loop dims per side each product is at most p,
        // otherwise it is bounded by p to the number of mapped tensor dims
        for (size_t e = 0; e < g->E.size(); e++) {
            const pase_edge_desc &d = g->E[e];
            uint32_t ms = 0, md = 0, ns = 0, nd = 0;
            bool distinct = true;
            for (uint32_t t = 0; t < d.rank; t++) {
                if (d.src_dim[t] >= 0) {
                    distinct &= !((ms >> d.src_dim[t]) & 1u);
                    ms |= 1u << d.src_dim[t];
                    ns++;
                }
                if (d.dst_dim[t] >= 0) {
                    distinct &= !((md >> d.dst_dim[t]) & 1u);
                    md |= 1u << d.dst_dim[t];
                    nd++;
                }
            }
            unsigned __int128 q = 1;
            for (uint32_t k = 0; k < (distinct ? 2u : ns + nd); k++) q *= p;
            if (q >= ((unsigned __int128)1 << 32))
                return fail(g, PASE_ERR_INVALID_ARGUMENT,
                            "volume model: tensor dims mapped to one loop dim make the device fractions too fine");
        }
    }
    const size_t nv = g->V.size();
    g->K.assign(nv, 0);
    g->ex.assign(nv, nullptr);
    g->weight_n.assign(nv, 0);
    g->halo = g->halo_opt == 1;
    g->halo_n.assign(nv, {});
    g->flops.assign(nv, 0);
    g->keep_n.assign(nv, 0);
    g->maxL.assign(nv, 0);
    // the configurations of a vertex depend only on its dimension count
    std::vector<std::vector<uint8_t>> &by_dims = g->ex_rows;
    by_dims.assign(kMaxDims + 1, {});
    for (size_t v = 0; v < nv; v++) {
        const uint32_t d = g->V[v].ndims;
        std::vector<uint8_t> &rows = by_dims[d];
        if (rows.empty()) {
            // split tuples with product <= p in lexicographic order (dim 0
            // slowest), by the lexicographic successor: step the last dim whose
            // next factor (x2, or +1 with every integer) still fits beside the
            // dims before it, and reset the dims after it to 1
            std::vector<uint32_t> cur(d, 1);
            uint64_t cnt = 0;
            for (;;) {
                if (++cnt > 65535) return fail(g, PASE_ERR_TOO_LARGE, "more than 65535 configurations");
                for (uint32_t x : cur) {
                    uint32_t code = x;
                    if (!factors) for (code = 0; (1u << code) < x; code++) {}
                    rows.push_back((uint8_t)code);
                }
                uint64_t prefix[kMaxDims + 1];
                prefix[0] = 1;
                for (uint32_t k = 0; k < d; k++) prefix[k + 1] = prefix[k] * cur[k];
                int k = (int)d - 1;
                for (; k >= 0; k--) {
                    const uint64_t next = factors ? cur[k] + 1ull : 2ull * cur[k];
                    if (prefix[k] * next <= p) break;
                }
                if (k < 0) break;
                cur[k] = factors ? cur[k] + 1 : 2 * cur[k];
                for (uint32_t j = k + 1; j < d; j++) cur[j] = 1;
            }
        }
        uint64_t K = rows.size() / d;
        if (K > 65535) return fail(g, PASE_ERR_TOO_LARGE, "more than 65535 configurations");
        g->K[v] = (uint32_t)K;
        g->ex[v] = &rows;
        uint64_t fl = g->V[v].flops_per_point, keep = 1;
        for (uint32_t k = 0; k < d; k++) {
            if (!mul_ok(fl, g->V[v].size[k], &fl))
                return fail(g, PASE_ERR_OVERFLOW, "layer FLOPs exceed 64 bits");
            if (!((g->V[v].reduce_mask >> k) & 1u) && !mul_ok(keep, g->V[v].size[k], &keep))
                return fail(g, PASE_ERR_OVERFLOW, "layer size exceeds 64 bits");
        }
        if (fl >> 62 || keep >> 62) return fail(g, PASE_ERR_OVERFLOW, "layer cost exceeds 2^62");
        g->flops[v] = fl;
        g->keep_n[v] = keep;
        // t_l <= flops + r * (p - 1) * keep (+ r * 2 * weight words with the gradient term)
        uint64_t comm, m;
        if (!mul_ok(g->r, (uint64_t)(p - 1), &comm) || !mul_ok(comm, keep, &comm) || !add_ok(fl, comm, &m))
            return fail(g, PASE_ERR_OVERFLOW, "layer cost exceeds 64 bits");
        if (g->grad_opt && g->V[v].weight_mask && g->V[v].weight_per_point) {
            uint64_t w = g->V[v].weight_per_point, gr;
            for (uint32_t k = 0; k < d; k++)
                if (((g->V[v].weight_mask >> k) & 1u) && !mul_ok(w, g->V[v].size[k], &w))
                    return fail(g, PASE_ERR_OVERFLOW, "weight tensor exceeds 64 bits");
            if (w >> 60 || !mul_ok(g->r, 2 * w, &gr) || !add_ok(m, gr, &m))
                return fail(g, PASE_ERR_OVERFLOW, "layer cost exceeds 64 bits");
            g->weight_n[v] = w;
        }
        g->halo_n[v].fill(0);
        if (g->halo) {
            // halo term: per halo dim k, I_k = prod of the other input dims'
            // sizes; t_l grows by at most r * 2 * halo[k] * I_k per dim
            const pase_vertex_desc &vd = g->V[v];
            for (uint32_t k = 0; k < d; k++) {
                if (!vd.halo[k]) continue;
                uint64_t I = 1, hw;
                for (uint32_t j = 0; j < d; j++)
                    if (j != k && ((vd.input_mask >> j) & 1u) && !mul_ok(I, vd.size[j], &I))
                        return fail(g, PASE_ERR_OVERFLOW, "input tensor exceeds 64 bits");
                if (I >> 62 || !mul_ok(2ull * vd.halo[k], I, &hw) || !mul_ok(g->r, hw, &hw) || !add_ok(m, hw, &m))
                    return fail(g, PASE_ERR_OVERFLOW, "layer cost exceeds 64 bits");
                g->halo_n[v][k] = I;
            }
        }
        g->maxL[v] = m;
    }
    g->maxR.assign(g->E.size(), 0);
    for (size_t e = 0; e < g->E.size(); e++) {
        // the volume model moves at most the whole tensor in each direction
        const uint64_t words = g->E[e].elems * (g->volume ? 2 : 1);
        if (g->E[e].elems >> 61 || !mul_ok(g->r, words, &g->maxR[e]))
            return fail(g, PASE_ERR_OVERFLOW, "transfer cost exceeds 64 bits");
        if (g->volume) {
            g->mat_off[e] = g->mat_total;
            g->mat_total += (uint64_t)g->K[g->E[e].src] * g->K[g->E[e].dst];
            g->mat_row0[e] = g->mat_rows;
            g->mat_rows += g->K[g->E[e].src];
        }
    }
    g->enumerated = true;
    g->plan_wide = false;
    const pase_status st = plan_search(g, true);
    if (st != PASE_OK) { g->enumerated = false; return st; }
    g->planned = true;
    return PASE_OK;
}

extern "C" pase_status pase_num_configs(pase_graph_t g, uint32_t v, uint32_t *k) {
    if (!g || !k) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->enumerated) return fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    if (v >= g->V.size()) return fail(g, PASE_ERR_INVALID_ARGUMENT, "vertex id out of range");
    *k = g->K[v];
    return PASE_OK;
}

extern "C" pase_status pase_config_splits(pase_graph_t g, uint32_t v, uint32_t idx, uint32_t *splits) {
    if (!g || !splits) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->enumerated) return fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    if (v >= g->V.size() || idx >= g->K[v]) return fail(g, PASE_ERR_INVALID_ARGUMENT, "bad id");
    const uint32_t d = g->V[v].ndims;
    for (uint32_t k = 0; k < d; k++) {
        const uint32_t x = (*g->ex[v])[(size_t)idx * d + k];
        splits[k] = g->factors ? x : 1u << x;
    }
    return PASE_OK;
}

extern "C" pase_status pase_get_sequence(pase_graph_t g, uint32_t *order) {
    if (!g || !order) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->planned) return fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    for (size_t i = 0; i < g->plan.seq.size(); i++) order[i] = (uint32_t)g->plan.seq[i];
    return PASE_OK;
}

extern "C" pase_status pase_get_dependent_set(pase_graph_t g, uint32_t v, uint32_t *out, uint32_t cap,
                                              uint32_t *n) {
    if (!g || !n || (cap && !out)) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->planned) return fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    if (v >= g->V.size()) return fail(g, PASE_ERR_INVALID_ARGUMENT, "vertex id out of range");
    const auto &D = g->plan.v[g->plan.pos[v]].D;
    if (D.size() > cap) return fail(g, PASE_ERR_TOO_LARGE, "output array too small");
    for (size_t k = 0; k < D.size(); k++) out[k] = (uint32_t)D[k];
    *n = (uint32_t)D.size();
    return PASE_OK;
}

extern "C" pase_status pase_set_option(pase_graph_t g, pase_option opt, uint64_t value) {
    if (!g) return PASE_ERR_INVALID_ARGUMENT;
    switch (opt) {
    case PASE_OPT_KEEP_TABLES: g->keep_tables = value != 0; break;
    case PASE_OPT_MEMORY_BUDGET: g->mem_budget = value; break;
    case PASE_OPT_KERNEL:
        if (value > 1) return fail(g, PASE_ERR_INVALID_ARGUMENT, "kernel mode 0 or 1");
        g->kernel_mode = (int)value;
        break;
    case PASE_OPT_KEY_TYPE:
        if (value > 2) return fail(g, PASE_ERR_INVALID_ARGUMENT, "key type 0, 1 or 2");
        g->key_mode = (int)value;
        break;
    case PASE_OPT_PROFILE:
        if (value > 2) return fail(g, PASE_ERR_INVALID_ARGUMENT, "profile 0, 1 or 2");
        g->profile = (int)value;
        break;
    case PASE_OPT_SCHEDULE:
        if (value != kSchedLevel && value != kSchedSeq && value != kSchedBulk && value != kSchedSplit)
            return fail(g, PASE_ERR_INVALID_ARGUMENT, "schedule 0, 1, 4 or 5");
        g->schedule = (int)value;
        break;
    case PASE_OPT_TILE_COLS:
        if (value != 0 && std::find(std::begin(kTZ), std::end(kTZ), value) == std::end(kTZ))
            return fail(g, PASE_ERR_INVALID_ARGUMENT, "tile columns 0, 8, 12, 14, 16, 24 or 28");
        g->tile_cols = (uint32_t)value;
        break;
    case PASE_OPT_TILE_ROWS:
        if (value > 2) return fail(g, PASE_ERR_INVALID_ARGUMENT, "tile rows 0, 1 or 2");
        g->tile_rows = (uint32_t)value;
        break;
    case PASE_OPT_TILE_PARTS:
        if (value != 0 && value != 1 && value != 2 && value != 4)
            return fail(g, PASE_ERR_INVALID_ARGUMENT, "tile parts 0, 1, 2 or 4");
        g->tile_parts = (uint32_t)value;
        break;
    case PASE_OPT_ORDER:
        if (value > 1) return fail(g, PASE_ERR_INVALID_ARGUMENT, "order 0 or 1");
        g->order_mode = (int)value;
        break;
    case PASE_OPT_DIRECT_CELLS:
        g->direct_cells = value;
        break;
    case PASE_OPT_BULK_US:
        if (value > 1000000000ull) return fail(g, PASE_ERR_INVALID_ARGUMENT, "bulk threshold <= 1e9 us");
        g->bulk_us = (uint32_t)value;
        break;
    case PASE_OPT_HALO:
        if (value > 1) return fail(g, PASE_ERR_INVALID_ARGUMENT, "halo 0 or 1");
        g->halo_opt = (uint32_t)value;
        break;
    case PASE_OPT_GRAD_SYNC:
        if (value > 1) return fail(g, PASE_ERR_INVALID_ARGUMENT, "grad sync 0 or 1");
        g->grad_opt = (uint32_t)value;
        break;
    case PASE_OPT_TRANSFER:
        if (value > 1) return fail(g, PASE_ERR_INVALID_ARGUMENT, "transfer model 0 or 1");
        g->transfer_opt = (uint32_t)value;
        break;
    case PASE_OPT_CONFIG_SET:
        if (value > 1) return fail(g, PASE_ERR_INVALID_ARGUMENT, "config set 0 or 1");
        g->config_set = (uint32_t)value;
        break;
    case PASE_OPT_C_SPLITS:
        if (value > 65535) return fail(g, PASE_ERR_INVALID_ARGUMENT, "c splits 0..65535");
        g->c_splits = (uint32_t)value;
        break;
    case PASE_OPT_FUSED_MIN:
        if (value > 1) return fail(g, PASE_ERR_INVALID_ARGUMENT, "fused minimum 0 or 1");
        g->fuse_min = value != 0;
        break;
    case PASE_OPT_HOIST_ELEMS:
        g->hoist_elems = value;
        break;
    default: return fail(g, PASE_ERR_INVALID_ARGUMENT, "unknown option");
    }
    // options that change the plan need a fresh enumeration
    if ((opt == PASE_OPT_KEEP_TABLES || opt == PASE_OPT_KERNEL || opt == PASE_OPT_MEMORY_BUDGET ||
         opt == PASE_OPT_SCHEDULE || opt == PASE_OPT_TILE_COLS || opt == PASE_OPT_TILE_ROWS ||
         opt == PASE_OPT_TILE_PARTS || opt == PASE_OPT_C_SPLITS || opt == PASE_OPT_ORDER ||
         opt == PASE_OPT_DIRECT_CELLS || opt == PASE_OPT_BULK_US || opt == PASE_OPT_KEY_TYPE ||
         opt == PASE_OPT_FUSED_MIN || opt == PASE_OPT_HOIST_ELEMS) &&
        g->enumerated) {
        g->searched = false;
        const pase_status st = plan_search(g, true);
        g->planned = st == PASE_OK;
        if (st != PASE_OK) return st;
    }
    return PASE_OK;
}

extern "C" pase_status pase_override_costs(pase_graph_t g, const uint64_t *layer, const uint64_t *edge) {
    if (!g || !layer || (!edge && !g->E.empty())) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->planned) return fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    const size_t nv = g->V.size(), ne = g->E.size();
    std::vector<uint64_t> old_layer = g->ov_layer, old_layer_off = g->ov_layer_off, old_edge = g->ov_edge,
                          old_edge_off = g->ov_edge_off;
    const bool was = g->overridden;
    g->ov_layer_off.assign(nv, 0);
    uint64_t tot = 0;
    for (size_t v = 0; v < nv; v++) { g->ov_layer_off[v] = tot; tot += g->K[v]; }
    g->ov_layer.assign(layer, layer + tot);
    g->ov_edge_off.assign(ne, 0);
    tot = 0;
    for (size_t e = 0; e < ne; e++) {
        g->ov_edge_off[e] = tot;
        tot += (uint64_t)g->K[g->E[e].src] * g->K[g->E[e].dst];
    }
    g->ov_edge.assign(edge ? edge : layer, edge ? edge + tot : layer);
    g->overridden = true;
    g->searched = false;
    const pase_status st = plan_search(g, false);
    if (st != PASE_OK) {
        // back to the plan of the costs before this call (which was valid)
        const std::string msg = g->err;
        g->overridden = false;
        g->ov_layer.swap(old_layer);
        g->ov_layer_off.swap(old_layer_off);
        g->ov_edge.swap(old_edge);
        g->ov_edge_off.swap(old_edge_off);
        g->overridden = was;
        g->planned = plan_search(g, false) == PASE_OK;
        g->err = msg;
        return st;
    }
    return PASE_OK;
}

extern "C" pase_status pase_workspace_size(pase_graph_t g, uint64_t *bytes) {
    if (!g || !bytes) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->planned) return fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    *bytes = g->plan.total;
    return PASE_OK;
}

extern "C" pase_status pase_set_workspace(pase_graph_t g, void *device_ptr, uint64_t bytes) {
    if (!g) return PASE_ERR_INVALID_ARGUMENT;
    if (device_ptr && ((uintptr_t)device_ptr % 256))
        return fail(g, PASE_ERR_INVALID_ARGUMENT, "workspace must be 256-byte aligned");
    g->lent_ws = device_ptr;
    g->lent_bytes = device_ptr ? bytes : 0;
    g->searched = false;
    return PASE_OK;
}

extern "C" pase_status pase_find_best_strategy(pase_graph_t g, void *stream, uint64_t *min_cost,
                                               uint32_t *config_idx) {
    if (!g || !min_cost || !config_idx) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->planned) return fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    if (g->lent_ws && g->lent_bytes < g->plan.total)
        return fail(g, PASE_ERR_OUT_OF_MEMORY, "lent workspace smaller than pase_workspace_size");
    return device_search(g, stream, min_cost, config_idx);
}

extern "C" pase_status pase_plan_check(pase_graph_t g, uint64_t *image_bytes) {
    if (!g || !image_bytes) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->planned) return fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    return plan_check(g, image_bytes);
}

extern "C" pase_status pase_find_best_strategy_noalloc(pase_graph_t g, void *stream, uint64_t *min_cost,
                                                       uint32_t *config_idx) {
    if (!g || !min_cost || !config_idx) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->planned) return fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    return device_search_noalloc(g, stream, min_cost, config_idx);
}

static pase_status find_entry(pase_graph_t g, uint32_t v, const uint32_t *dep_cfg, int *pos,
                              uint64_t *idx) {
    if (!g->searched) return fail(g, PASE_ERR_BAD_STATE, "no search has run");
    if (v >= g->V.size()) return fail(g, PASE_ERR_INVALID_ARGUMENT, "vertex id out of range");
    const VPlan &vp = g->plan.v[g->plan.pos[v]];
    uint64_t x = 0;
    for (size_t k = 0; k < vp.layout.size(); k++) {
        size_t at = std::lower_bound(vp.D.begin(), vp.D.end(), vp.layout[k]) - vp.D.begin();
        uint32_t c = dep_cfg[at];
        if (c >= g->K[vp.layout[k]]) return fail(g, PASE_ERR_INVALID_ARGUMENT, "config out of range");
        x += c * vp.stride[k];
    }
    *pos = g->plan.pos[v];
    *idx = x;
    return PASE_OK;
}

extern "C" pase_status pase_table_entry(pase_graph_t g, uint32_t v, const uint32_t *dep_cfg,
                                        uint64_t *cost, uint32_t *argmin) {
    if (!g || !cost || !argmin) return PASE_ERR_INVALID_ARGUMENT;
    if (v < g->V.size() && g->planned && !g->plan.v[g->plan.pos[v]].D.empty() && !dep_cfg)
        return PASE_ERR_INVALID_ARGUMENT;
    int pos;
    uint64_t idx;
    pase_status st = find_entry(g, v, dep_cfg, &pos, &idx);
    if (st != PASE_OK) return st;
    if (!g->keep_tables && pos != (int)g->plan.v.size() - 1)
        return fail(g, PASE_ERR_BAD_STATE, "tables are not kept (PASE_OPT_KEEP_TABLES)");
    return device_table_entry(g, pos, idx, cost, argmin);
}

extern "C" pase_status pase_table_fingerprint(pase_graph_t g, uint32_t v, uint64_t *fp_cost,
                                              uint64_t *fp_arg) {
    if (!g || !fp_cost || !fp_arg) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->searched) return fail(g, PASE_ERR_BAD_STATE, "no search has run");
    if (v >= g->V.size()) return fail(g, PASE_ERR_INVALID_ARGUMENT, "vertex id out of range");
    int pos = g->plan.pos[v];
    if (!g->keep_tables && pos != (int)g->plan.v.size() - 1)
        return fail(g, PASE_ERR_BAD_STATE, "tables are not kept (PASE_OPT_KEEP_TABLES)");
    return device_fingerprint(g, pos, fp_cost, fp_arg);
}

extern "C" pase_status pase_layer_costs(pase_graph_t g, uint32_t v, uint64_t *out) {
    if (!g || !out) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->searched) return fail(g, PASE_ERR_BAD_STATE, "no search has run");
    if (v >= g->V.size()) return fail(g, PASE_ERR_INVALID_ARGUMENT, "vertex id out of range");
    return device_layer_costs(g, v, out);
}

extern "C" pase_status pase_edge_costs(pase_graph_t g, uint32_t e, uint64_t *out) {
    if (!g || !out) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->searched) return fail(g, PASE_ERR_BAD_STATE, "no search has run");
    if (e >= g->E.size()) return fail(g, PASE_ERR_INVALID_ARGUMENT, "edge id out of range");
    return device_edge_costs(g, e, out);
}

extern "C" pase_status pase_stats(pase_graph_t g, pase_run_stats *out) {
    if (!g || !out) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->searched) return fail(g, PASE_ERR_BAD_STATE, "no search has run");
    *out = g->stats;
    return PASE_OK;
}

extern "C" pase_status pase_vertex_info_get(pase_graph_t g, uint32_t v, pase_vertex_info *out) {
    if (!g || !out) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->planned) return fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    if (v >= g->V.size()) return fail(g, PASE_ERR_INVALID_ARGUMENT, "vertex id out of range");
    const VPlan &vp = g->plan.v[g->plan.pos[v]];
    pase_vertex_info x;
    std::memset(&x, 0, sizeof x);
    x.position = (uint32_t)g->plan.pos[v];
    x.kernel = (uint32_t)vp.kernel;
    x.num_configs = vp.K;
    x.dep_count = (uint32_t)vp.D.size();
    x.entries = vp.N;
    x.cells = vp.N * vp.K;
    x.column = vp.kernel == kRows ? vp.z : -1;
    x.outer = (uint32_t)vp.MO;
    x.rows = (uint32_t)vp.MR;
    x.tile_cols = vp.TZ;
    x.tile_rows = vp.TM;
    x.parts = vp.kernel == kRows ? vp.parts : 0;
    x.splits = vp.nsplit;
    x.row_terms = vp.na;
    x.lookups = (uint32_t)vp.terms.size();
    x.fill_ms = vp.fill_ms;
    x.level = (uint32_t)vp.level;
    x.lane = (uint32_t)vp.lane;
    std::vector<uint64_t> qmax, tmax;
    if (cost_bounds(g, &qmax, &tmax)) {
        x.key_bound = qmax[x.position];
        x.table_bound = tmax[x.position];
    } else {
        x.key_bound = x.table_bound = ~0ull;
    }
    x.key_type = g->plan_key_type;
    x.fused = vp.fuse_into >= 0 ? 1u : vp.fused_from >= 0 ? 2u : 0u;
    x.prep_after = vp.prep_after;
    x.prep_lane = (uint32_t)vp.prep_lane;
    *out = x;
    return PASE_OK;
}
