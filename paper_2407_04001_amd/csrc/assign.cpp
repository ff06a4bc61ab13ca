// Greedy device assignment of a chosen strategy (Sec. II, the device
// assignment paragraph after the cost model): the search prices a strategy
// with a fixed numbering of each configuration's parts; afterwards every
// vertex's parts are placed on devices so that a part lands where the parts
// of its already placed neighbours hold the most of the tensors they share.
//
// Host code: the work is a short chain of vertices, each a few thousand
// (part, device) pairs at most, well below the cost of one kernel launch.
//
// Geometry.  A configuration with splits s over loop dims cuts each loop dim k
// into s_k equal fractions; part g is the mixed-radix grid point of g (loop
// dim 0 slowest).  A tensor dim t of an edge mapped to loop dim a at the
// source and b at the destination is, at the source, the fraction interval
// [x_a / s_a, (x_a + 1) / s_a) (the whole dim when unmapped), at the
// destination likewise with the destination's split.  In units of
// 1 / (s_a * s'_b) the source interval is [x_a s'_b, (x_a + 1) s'_b) and the
// destination's [y_b s_a, (y_b + 1) s_a); the shared length is the overlap of
// the two integer intervals.  The shared elements of two parts are
// floor(elems * prod_t shared_t / prod_t (s_a s'_b)).
#include <algorithm>
#include <chrono>
#include <cstring>
#include <vector>

#include "internal.h"

namespace {

using u128 = unsigned __int128;

struct EdgeGeom {
    // per tensor dim: split at the source side (1 unmapped), at the destination
    // side, and the loop dim each maps to (-1 unmapped)
    uint32_t rank = 0;
    uint64_t a[PASE_MAX_DIMS], b[PASE_MAX_DIMS];
    int la[PASE_MAX_DIMS], lb[PASE_MAX_DIMS];
    u128 cells = 1;     // prod_t a_t * b_t
    u128 src_part = 1;  // cells one source part covers: prod_t b_t
    u128 dst_part = 1;  // cells one destination part covers: prod_t a_t
};

// Grid point of part g of splits s (d loop dims), loop dim 0 slowest.
void grid_point(const uint32_t *s, uint32_t d, uint64_t g, uint64_t *x) {
    for (uint32_t k = d; k-- > 0;) {
        x[k] = g % s[k];
        g /= s[k];
    }
}

// Shared cells of the source part at grid point xs and the destination part at xd.
u128 shared_cells(const EdgeGeom &G, const uint64_t *xs, const uint64_t *xd) {
    u128 c = 1;
    for (uint32_t t = 0; t < G.rank; t++) {
        const uint64_t ps = G.la[t] >= 0 ? xs[G.la[t]] : 0, pd = G.lb[t] >= 0 ? xd[G.lb[t]] : 0;
        const uint64_t lo = std::max(ps * G.b[t], pd * G.a[t]);
        const uint64_t hi = std::min((ps + 1) * G.b[t], (pd + 1) * G.a[t]);
        if (hi <= lo) return 0;
        c *= hi - lo;
    }
    return c;
}

// floor(elems * c / cells) for 0 < c <= cells < 2^64; 64-bit division when
// the product fits (the 128-bit one is several times slower)
uint64_t share(uint64_t elems, u128 c, u128 cells) {
    if (c == cells) return elems;
    const u128 num = (u128)elems * c;
    if (!(num >> 64)) return (uint64_t)num / (uint64_t)cells;
    return (uint64_t)(num / cells);
}

}  // namespace

extern "C" pase_status pase_assign_devices(pase_graph_t g, const uint32_t *config_idx, int32_t *devices,
                                           uint64_t *edge_locality, uint64_t *edge_xfer) {
    if (!g || !config_idx || !devices) return PASE_ERR_INVALID_ARGUMENT;
    if (!g->enumerated) return pase::fail(g, PASE_ERR_BAD_STATE, "configurations not enumerated");
    const auto t0 = std::chrono::steady_clock::now();
    const uint32_t nv = (uint32_t)g->V.size(), ne = (uint32_t)g->E.size(), p = g->p;
    if (p > pase::kAssignMaxDevices)
        return pase::fail(g, PASE_ERR_TOO_LARGE, "device assignment needs p <= 1024");

    // splits and part counts of the strategy
    std::vector<uint32_t> S((size_t)nv * PASE_MAX_DIMS, 1);
    std::vector<uint64_t> parts(nv, 1);
    for (uint32_t v = 0; v < nv; v++) {
        if (config_idx[v] >= g->K[v]) return pase::fail(g, PASE_ERR_INVALID_ARGUMENT, "configuration out of range");
        const uint32_t d = g->V[v].ndims;
        for (uint32_t k = 0; k < d; k++) {
            const uint32_t x = (*g->ex[v])[(size_t)config_idx[v] * d + k];
            S[(size_t)v * PASE_MAX_DIMS + k] = g->factors ? x : 1u << x;
            parts[v] *= S[(size_t)v * PASE_MAX_DIMS + k];
        }
    }
    std::vector<EdgeGeom> geom(ne);
    std::vector<uint64_t> elems_sum(nv, 0);
    for (uint32_t e = 0; e < ne; e++) {
        const pase_edge_desc &ed = g->E[e];
        EdgeGeom &G = geom[e];
        G.rank = ed.rank;
        for (uint32_t t = 0; t < ed.rank; t++) {
            G.la[t] = ed.src_dim[t];
            G.lb[t] = ed.dst_dim[t];
            G.a[t] = G.la[t] >= 0 ? S[(size_t)ed.src * PASE_MAX_DIMS + G.la[t]] : 1;
            G.b[t] = G.lb[t] >= 0 ? S[(size_t)ed.dst * PASE_MAX_DIMS + G.lb[t]] : 1;
            G.cells *= (u128)G.a[t] * G.b[t];
            G.src_part *= G.b[t];
            G.dst_part *= G.a[t];
            // several tensor dims on one loop dim multiply its split: keep the
            // cell count (and so every product below) within 64 bits
            if (G.cells >> 64)
                return pase::fail(g, PASE_ERR_TOO_LARGE, "an edge's splits cut its tensor into 2^64 cells or more");
        }
        // a vertex's localities sum the tensors of its edges: keep them in 64 bits
        for (uint32_t w : {ed.src, ed.dst})
            if (__builtin_add_overflow(elems_sum[w], ed.elems, &elems_sum[w]))
                return pase::fail(g, PASE_ERR_OVERFLOW, "tensor elements of a vertex's edges exceed 64 bits");
    }
    std::vector<std::vector<uint32_t>> incident(nv);
    for (uint32_t e = 0; e < ne; e++) {
        incident[g->E[e].src].push_back(e);
        incident[g->E[e].dst].push_back(e);
    }

    // dev[v][d] = part of v on device d (-1 none); the first vertex keeps the grid numbering
    std::vector<int32_t> dev((size_t)nv * p, -1);
    for (uint64_t q = 0; q < parts[0]; q++) dev[q] = (int32_t)q;
    struct Pair {
        uint64_t w;
        uint32_t part, device;
    };
    std::vector<Pair> pairs;
    std::vector<uint64_t> W;
    std::vector<uint32_t> touched;   // entries of W that are nonzero
    std::vector<char> part_done(p), dev_used(p);
    for (uint32_t v = 1; v < nv; v++) {
        const uint64_t P = parts[v];
        const uint32_t dv = g->V[v].ndims;
        const uint32_t *sv = &S[(size_t)v * PASE_MAX_DIMS];
        W.assign((size_t)P * p, 0);
        touched.clear();
        for (uint32_t e : incident[v]) {
            const pase_edge_desc &ed = g->E[e];
            const bool v_is_src = ed.src == v;
            const uint32_t other = v_is_src ? ed.dst : ed.src;
            if (other > v) continue;   // not placed yet
            const EdgeGeom &G = geom[e];
            const uint64_t *fv = v_is_src ? G.a : G.b, *fo = v_is_src ? G.b : G.a;
            const int *lv = v_is_src ? G.la : G.lb, *lo = v_is_src ? G.lb : G.la;
            for (uint32_t d = 0; d < p; d++) {
                const int32_t h = dev[(size_t)other * p + d];
                if (h < 0) continue;
                uint64_t xo[PASE_MAX_DIMS], xlo[PASE_MAX_DIMS], xhi[PASE_MAX_DIMS], x[PASE_MAX_DIMS];
                grid_point(&S[(size_t)other * PASE_MAX_DIMS], g->V[other].ndims, (uint64_t)h, xo);
                // digits of v's parts that can share cells with the other part: per
                // tensor dim mapped at v, the fractions [y / f_v, (y + 1) / f_v) that
                // meet [x_o / f_o, (x_o + 1) / f_o)
                for (uint32_t k = 0; k < dv; k++) xlo[k] = 0, xhi[k] = sv[k];
                for (uint32_t t = 0; t < G.rank; t++) {
                    if (lv[t] < 0) continue;
                    const uint64_t po = lo[t] >= 0 ? xo[lo[t]] : 0;
                    const uint64_t a = po * fv[t] / fo[t], b = ((po + 1) * fv[t] + fo[t] - 1) / fo[t];
                    xlo[lv[t]] = std::max(xlo[lv[t]], a);
                    xhi[lv[t]] = std::min(xhi[lv[t]], b);
                }
                bool empty = false;
                for (uint32_t k = 0; k < dv; k++) empty |= xlo[k] >= xhi[k];
                if (empty) continue;
                for (uint32_t k = 0; k < dv; k++) x[k] = xlo[k];
                for (;;) {
                    uint64_t q = 0;
                    for (uint32_t k = 0; k < dv; k++) q = q * sv[k] + x[k];
                    const u128 c = v_is_src ? shared_cells(G, x, xo) : shared_cells(G, xo, x);
                    if (c) {
                        const uint64_t w = share(ed.elems, c, G.cells);
                        uint64_t &slot = W[q * p + d];
                        if (w && !slot) touched.push_back((uint32_t)(q * p + d));
                        slot += w;
                    }
                    uint32_t k = dv;   // next digit tuple, last loop dim fastest
                    while (k-- > 0) {
                        if (++x[k] < xhi[k]) break;
                        x[k] = xlo[k];
                    }
                    if (k == UINT32_MAX) break;
                }
            }
        }
        // greedy matching: pairs by locality descending, ties to the lower part, then
        // the lower device; a pair is taken when both its part and its device are
        // free.  Pairs of locality 0 come last in (part, device) order: the lowest
        // free part takes the lowest free device, and so on
        pairs.clear();
        for (uint32_t i : touched) pairs.push_back({W[i], (uint32_t)(i / p), (uint32_t)(i % p)});
        std::sort(pairs.begin(), pairs.end(), [](const Pair &x, const Pair &y) {
            if (x.w != y.w) return x.w > y.w;
            if (x.part != y.part) return x.part < y.part;
            return x.device < y.device;
        });
        std::fill(part_done.begin(), part_done.end(), 0);
        std::fill(dev_used.begin(), dev_used.end(), 0);
        uint64_t placed = 0;
        for (const Pair &x : pairs) {
            if (part_done[x.part] || dev_used[x.device]) continue;
            part_done[x.part] = dev_used[x.device] = 1;
            dev[(size_t)v * p + x.device] = (int32_t)x.part;
            ++placed;
        }
        for (uint32_t q = 0, d = 0; q < P && placed < P; q++) {
            if (part_done[q]) continue;
            while (dev_used[d]) d++;
            dev_used[d] = 1;
            dev[(size_t)v * p + d] = (int32_t)q;
            ++placed;
        }
    }

    // locality and r * t_x of every edge under the assignment: per device the
    // destination needs its part minus what the source's part there already
    // holds (forward), the source likewise (backward); t_x takes the largest
    // per direction, words rounded up
    for (uint32_t e = 0; e < ne; e++) {
        const pase_edge_desc &ed = g->E[e];
        const EdgeGeom &G = geom[e];
        uint64_t xs[PASE_MAX_DIMS], xd[PASE_MAX_DIMS], loc = 0;
        u128 fwd = 0, bwd = 0;
        for (uint32_t d = 0; d < p; d++) {
            const int32_t hs = dev[(size_t)ed.src * p + d], hd = dev[(size_t)ed.dst * p + d];
            u128 c = 0;
            if (hs >= 0 && hd >= 0) {
                grid_point(&S[(size_t)ed.src * PASE_MAX_DIMS], g->V[ed.src].ndims, (uint64_t)hs, xs);
                grid_point(&S[(size_t)ed.dst * PASE_MAX_DIMS], g->V[ed.dst].ndims, (uint64_t)hd, xd);
                c = shared_cells(G, xs, xd);
                if (c) loc += share(ed.elems, c, G.cells);
            }
            if (hd >= 0) fwd = std::max(fwd, G.dst_part - c);
            if (hs >= 0) bwd = std::max(bwd, G.src_part - c);
        }
        const u128 E = ed.elems;
        const u128 words = (E * fwd + G.cells - 1) / G.cells + (E * bwd + G.cells - 1) / G.cells;
        uint64_t x;
        if ((words >> 64) || __builtin_mul_overflow((uint64_t)words, g->r, &x))
            return pase::fail(g, PASE_ERR_OVERFLOW, "transfer cost under the assignment exceeds 64 bits");
        if (edge_locality) edge_locality[e] = loc;
        if (edge_xfer) edge_xfer[e] = x;
    }
    std::memcpy(devices, dev.data(), dev.size() * sizeof(int32_t));
    g->stats.assign_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    return PASE_OK;
}
