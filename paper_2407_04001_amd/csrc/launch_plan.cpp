// Host planning of one search's launches (no HIP calls, so that it runs and
// is checked without a GPU): kernel descriptors of every position resolved
// against the workspace base, the batched launches of each launch slot, and
// the constant-region image the device runtime uploads before the first
// kernel.
#include <algorithm>
#include <cstring>
#include <map>
#include <type_traits>

#include "launch.h"

namespace pase {

static uint32_t grid_for(uint64_t n, uint32_t block = 256, uint32_t cap = 8192) {
    uint64_t b = (n + block - 1) / block;
    return (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(b, cap));
}

static uint32_t plan_digit(const VPlan &vp, int vertex) {
    for (size_t k = 0; k < vp.layout.size(); k++)
        if (vp.layout[k] == vertex) return (uint32_t)k;
    return ~0u;
}

// Strides with which consumer position i reads table T_j: (stride of v_i, per plan digit).
static void lookup_strides(const Plan &P, int i, int j, uint32_t &sc, uint32_t sd[kMaxDep]) {
    const VPlan &vi = P.v[i], &vj = P.v[j];
    sc = 0;
    for (int k = 0; k < kMaxDep; k++) sd[k] = 0;
    for (size_t k = 0; k < vj.layout.size(); k++) {
        int u = vj.layout[k];
        if (u == vi.vi) sc = (uint32_t)vj.stride[k];
        else sd[plan_digit(vi, u)] = (uint32_t)vj.stride[k];
    }
}

// Largest element index a strided read can reach: (K-1)*sc + sum (radix-1)*stride.
static uint64_t max_index(uint32_t K, uint32_t sc, const uint32_t *sd, const uint32_t *rad, int m) {
    uint64_t x = (uint64_t)(K - 1) * sc;
    for (int k = 0; k < m; k++) x += (uint64_t)(rad[k] - 1) * sd[k];
    return x;
}

template <typename KeyT>
pase_status build_launches(pase_graph_t g, char *ws, std::vector<Launch<KeyT>> &out,
                           std::vector<Contrib> &contrib) {
    const Plan &P = g->plan;
    const int n = (int)P.v.size();
    out.assign(n, Launch<KeyT>());
    contrib.clear();
    const uint64_t *ovedge = (const uint64_t *)(ws + P.off_ovedge);
    for (int i = 0; i < n; i++) {
        const VPlan &vp = P.v[i];
        Launch<KeyT> &L = out[i];
        KeyT *blocks = (KeyT *)(ws + P.off_block + vp.block_off);
        std::memset(&L.prep, 0, sizeof L.prep);
        L.prep.blocks = blocks;
        L.prep.vi = (uint32_t)vp.vi;
        L.prep.K = vp.K;
        L.prep.bits = vp.bits;
        uint32_t rad[kMaxDep];
        for (size_t k = 0; k < vp.layout.size(); k++) rad[k] = g->K[vp.layout[k]];
        const int m = (int)vp.layout.size();
        bool bounds_ok = true;
        auto other_of = [&](int e) {
            return (int)g->E[e].src == vp.vi ? (int)g->E[e].dst : (int)g->E[e].src;
        };
        auto edge_contrib = [&](int e, uint32_t dig) {
            Contrib c;
            std::memset(&c, 0, sizeof c);
            bool is_src = (int)g->E[e].src == vp.vi;
            if (g->overridden || g->volume) {
                c.kind = kContribTable;
                c.raw_u64 = 1;
                c.ptr = g->overridden ? ovedge + g->ov_edge_off[e] : (const uint64_t *)(ws + P.off_vmat) + g->mat_off[e];
                uint32_t Kd = g->K[g->E[e].dst];
                if (is_src) { c.sc = Kd; c.sd[dig] = 1; }
                else { c.sc = 1; c.sd[dig] = Kd; }
                if (max_index(vp.K, c.sc, c.sd, rad, m) >= (uint64_t)g->K[g->E[e].src] * Kd)
                    bounds_ok = false;
            } else {
                c.kind = kContribEdge;
                c.edge = (uint32_t)e;
                c.dig = dig;
                c.vi_is_src = is_src;
            }
            contrib.push_back(c);
        };
        auto table_contrib = [&](const TermRef &t) {
            Contrib c;
            std::memset(&c, 0, sizeof c);
            c.kind = kContribTable;
            c.ptr = ws + P.off_T + P.v[t.j].T_off;
            lookup_strides(P, i, t.j, c.sc, c.sd);
            // the prep block only feeds digits of the lookup, so every index stays inside T_j
            if (max_index(vp.K, c.sc, c.sd, rad, m) >= P.v[t.j].N) bounds_ok = false;
            contrib.push_back(c);
        };
        auto layer_contrib = [&]() {
            Contrib c;
            std::memset(&c, 0, sizeof c);
            c.kind = kContribLayer;
            contrib.push_back(c);
        };
        uint64_t boff = 0;
        auto add_block = [&](const std::vector<int> &pre, int post, uint32_t ld, uint32_t cb) -> int {
            Block &bk = L.prep.blk[L.prep.nblocks];
            std::memset(&bk, 0, sizeof bk);
            bk.npre = (uint32_t)pre.size();
            uint64_t el = 1;
            for (size_t k = 0; k < pre.size(); k++) {
                bk.pre[k] = plan_digit(vp, pre[k]);
                bk.prerad[k] = g->K[pre[k]];
                el *= g->K[pre[k]];
            }
            bk.post = post >= 0 ? (int32_t)plan_digit(vp, post) : -1;
            bk.postrad = post >= 0 ? g->K[post] : 1;
            bk.ld = ld;
            bk.elems = el * vp.K * ld;
            bk.out_off = boff;
            boff += (bk.elems + 31) / 32 * 32;
            bk.c_begin = cb;
            bk.c_end = (uint32_t)contrib.size();
            bk.rows = (uint32_t)el;
            // a workgroup covers `span` runs of kPrepThreads elements, so that
            // the chain of scalar loads of the block's descriptors and
            // contributions is paid once per span; large blocks keep at
            // least ~4096 workgroups
            const uint64_t runs = ((uint64_t)vp.K * ld + kPrepThreads - 1) / kPrepThreads;
            bk.span = (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(8, runs * el / 4096));
            bk.chunks = (uint32_t)((runs + bk.span - 1) / bk.span);
            bk.wg_begin = L.prep.nwg;
            L.prep.nwg += bk.rows * bk.chunks;
            L.prep.total += bk.elems;
            return (int)L.prep.nblocks++;
        };
        if (vp.kernel == kDirect) {
            // every term over all plan digits; no blocks
            DirectArgs &da = L.da;
            std::memset(&da, 0, sizeof da);
            da.c_begin = (uint32_t)contrib.size();
            layer_contrib();
            for (int e : vp.edges) edge_contrib(e, plan_digit(vp, other_of(e)));
            for (const auto &t : vp.terms) table_contrib(t);
            da.c_end = (uint32_t)contrib.size();
            da.vi = (uint32_t)vp.vi;
            da.K = vp.K;
            da.bits = vp.bits;
            da.out_shift = vp.out_shift;
            da.m = (uint32_t)vp.layout.size();
            for (size_t k = 0; k < vp.layout.size(); k++) da.rad[k] = g->K[vp.layout[k]];
            // lanes per entry: enough threads to fill the GPU, at most a
            // workgroup (four waves, combined in LDS), at most K
            da.group_log2 = 0;
            while (da.group_log2 < 8 && (vp.N << da.group_log2) < 65536 && (2u << da.group_log2) <= vp.K)
                da.group_log2++;
            da.N = vp.N;
            da.T = ws + P.off_T + vp.T_off;
            da.A = (uint16_t *)(ws + P.off_A + vp.A_off);
            da.nblk = (uint32_t)std::min<uint64_t>(((vp.N << da.group_log2) + 255) / 256, 65535);
            L.direct = true;
        } else if (vp.kernel == kRows) {
            // column block B over (O..., c, z): everything not touching a row digit
            std::vector<int> OZ = vp.O;
            OZ.push_back(vp.z);
            auto in_oz = [&](int u) { return std::find(OZ.begin(), OZ.end(), u) != OZ.end(); };
            uint32_t cb = (uint32_t)contrib.size();
            layer_contrib();
            for (int e : vp.edges)
                if (in_oz(other_of(e))) edge_contrib(e, plan_digit(vp, other_of(e)));
            for (const auto &t : vp.terms) {
                bool all = true;
                for (int u : t.dig) all &= in_oz(u);
                if (all) table_contrib(t);
            }
            add_block(vp.O, vp.z, vp.ldz, cb);
            RowsArgs &ra = L.ra;
            std::memset(&ra, 0, sizeof ra);
            ra.B = blocks + L.prep.blk[0].out_off;
            // one-digit row blocks E_w, w in R
            for (size_t rk = 0; rk < vp.R.size(); rk++) {
                int w = vp.R[rk];
                cb = (uint32_t)contrib.size();
                for (int e : vp.edges)
                    if (other_of(e) == w) edge_contrib(e, plan_digit(vp, w));
                for (const auto &t : vp.terms)
                    if (t.dig.size() == 1 && t.dig[0] == w) table_contrib(t);
                if (contrib.size() == cb) continue;
                int b = add_block({}, w, g->K[w], cb);
                ATerm &at = ra.a[ra.na++];
                at.ptr = blocks + L.prep.blk[b].out_off;
                at.sc = g->K[w];
                at.bytes = (uint32_t)(L.prep.blk[b].elems * sizeof(KeyT));
                at.sdR[rk] = 1;
            }
            // lookups touching a row digit with two or more digits: read in the kernel
            for (const auto &t : vp.terms) {
                if (t.dig.size() < 2) continue;
                bool touches = false;
                for (int u : t.dig) touches |= std::count(vp.R.begin(), vp.R.end(), u) > 0;
                if (!touches) continue;
                if (ra.na >= (uint32_t)kMaxATerms) return fail(g, PASE_ERR_INTERNAL, "row terms");
                ATerm &at = ra.a[ra.na++];
                uint32_t sc, sd[kMaxDep];
                lookup_strides(P, i, t.j, sc, sd);
                if (max_index(vp.K, sc, sd, rad, m) >= P.v[t.j].N) bounds_ok = false;
                at.ptr = ws + P.off_T + P.v[t.j].T_off;
                at.sc = sc;
                at.bytes = (uint32_t)(P.v[t.j].N * 8);
                // plan digits: z (if there is a column digit), then O, then R
                const size_t zoff = vp.z >= 0 ? 1 : 0;
                for (size_t k = 0; k < vp.O.size(); k++) at.sdO[k] = sd[zoff + k];
                for (size_t k = 0; k < vp.R.size(); k++) at.sdR[k] = sd[zoff + vp.O.size() + k];
            }
            ra.ldz = vp.ldz;
            ra.Kz = vp.z >= 0 ? g->K[vp.z] : 1;
            ra.K = vp.K;
            ra.bits = vp.bits;
            ra.MO = (uint32_t)vp.MO;
            ra.MR = (uint32_t)vp.MR;
            ra.tiles_per_o = (uint32_t)((vp.MR + 64 * vp.TM - 1) / (64 * vp.TM));
            ra.nchunks = vp.nchunks;
            ra.nsplit = vp.nsplit;
            ra.cper = vp.cper;
            ra.nO = (uint32_t)vp.O.size();
            ra.nR = (uint32_t)vp.R.size();
            for (size_t k = 0; k < vp.O.size(); k++) ra.radO[k] = g->K[vp.O[k]];
            for (size_t k = 0; k < vp.R.size(); k++) ra.radR[k] = g->K[vp.R[k]];
            ra.T = ws + P.off_T + vp.T_off;
            ra.A = (uint16_t *)(ws + P.off_A + vp.A_off);
            ra.partial = ws + P.off_partial + vp.partial_off;
            ra.N = vp.N;
            ra.out_shift = vp.out_shift;
            // a workgroup takes 4 / parts tiles
            ra.parts = vp.parts;
            ra.total_tiles = (uint64_t)vp.nsplit * vp.nchunks * vp.MO * ra.tiles_per_o;
            uint64_t nbk = (ra.total_tiles + 4 / vp.parts - 1) / (4 / vp.parts);
            nbk = (nbk + 7) / 8 * 8;
            if (nbk > 0x7fffffffull) return fail(g, PASE_ERR_TOO_LARGE, "grid too large");
            ra.nblocks_launched = (uint32_t)nbk;
            L.rows = true;
            if (vp.nsplit > 1 || vp.fused_from >= 0) {
                L.red.nblk = grid_for(vp.N);
                L.red.partial = vp.fused_from >= 0 ? (void *)(ws + P.off_fused + vp.fkeys_off) : ra.partial;
                L.red.T = ra.T;
                L.red.A = ra.A;
                L.red.N = vp.N;
                L.red.nsplit = vp.nsplit;
                L.red.bits = vp.bits;
                L.red.out_shift = vp.out_shift;
            }
            if (vp.fused_from >= 0) {
                // the producer's epilogue forms this vertex's keys; its own fill
                // is the reduction of those keys (its row descriptor stays for
                // the producer to copy the row terms from)
                L.rows = false;
                L.fused = true;
                if (vp.nsplit != 1) return fail(g, PASE_ERR_INTERNAL, "fused minimum split over c");
            }
        } else {
            GenericArgs &ga = L.ga;
            std::memset(&ga, 0, sizeof ga);
            uint32_t cb = (uint32_t)contrib.size();
            layer_contrib();
            for (const auto &t : vp.terms)
                if (t.dig.empty()) table_contrib(t);
            int b0 = add_block({}, -1, 1, cb);
            GTerm &g0 = ga.t[ga.nt++];
            g0.ptr = blocks + L.prep.blk[b0].out_off;
            g0.sc = 1;
            for (int w : vp.D) {
                cb = (uint32_t)contrib.size();
                for (int e : vp.edges)
                    if (other_of(e) == w) edge_contrib(e, plan_digit(vp, w));
                for (const auto &t : vp.terms)
                    if (t.dig.size() == 1 && t.dig[0] == w) table_contrib(t);
                if (contrib.size() == cb) continue;
                int b = add_block({}, w, g->K[w], cb);
                GTerm &gt = ga.t[ga.nt++];
                gt.ptr = blocks + L.prep.blk[b].out_off;
                gt.sc = g->K[w];
                gt.sd[plan_digit(vp, w)] = 1;
            }
            for (const auto &t : vp.terms) {
                if (t.dig.size() < 2) continue;
                if (ga.nt >= (uint32_t)kMaxGTerms)
                    return fail(g, PASE_ERR_TOO_LARGE, "too many table lookups for one vertex");
                GTerm &gt = ga.t[ga.nt++];
                gt.ptr = ws + P.off_T + P.v[t.j].T_off;
                lookup_strides(P, i, t.j, gt.sc, gt.sd);
                if (max_index(vp.K, gt.sc, gt.sd, rad, m) >= P.v[t.j].N) bounds_ok = false;
            }
            ga.m = (uint32_t)vp.layout.size();
            ga.K = vp.K;
            ga.bits = vp.bits;
            // lanes per entry: enough threads to fill the GPU, at most one wave, at most K
            ga.group_log2 = 0;
            while (ga.group_log2 < 6 && (vp.N << ga.group_log2) < 65536 && (2u << ga.group_log2) <= vp.K)
                ga.group_log2++;
            for (size_t k = 0; k < vp.layout.size(); k++) ga.rad[k] = g->K[vp.layout[k]];
            ga.T = ws + P.off_T + vp.T_off;
            ga.A = (uint16_t *)(ws + P.off_A + vp.A_off);
            ga.N = vp.N;
            ga.out_shift = vp.out_shift;
            ga.nblk = (uint32_t)std::min<uint64_t>(((vp.N << ga.group_log2) + 255) / 256, 65535);
        }
        if (boff > vp.block_elems) return fail(g, PASE_ERR_INTERNAL, "block scratch overflow");
        if (!bounds_ok) return fail(g, PASE_ERR_INTERNAL, "a table lookup would leave its table");
        if (vp.nsplit > 1 && vp.partial_off + (uint64_t)vp.nsplit * vp.N * sizeof(KeyT) > P.partial_bytes)
            return fail(g, PASE_ERR_INTERNAL, "split scratch overflow");
        if (vp.block_off + boff * sizeof(KeyT) > P.block_bytes)
            return fail(g, PASE_ERR_INTERNAL, "block scratch overflow");
    }
    if (contrib.size() > P.contrib_count) return fail(g, PASE_ERR_INTERNAL, "contribution overflow");
    // fused minima: the producer's epilogue gets the reader's row terms other
    // than the producer's own table, and its column block
    for (int i1 = 0; i1 < n; i1++) {
        const int i2 = P.v[i1].fuse_into;
        if (i2 < 0) continue;
        if constexpr (sizeof(KeyT) != 8) {
            return fail(g, PASE_ERR_INTERNAL, "fused minimum with 128-bit keys");
        } else {
            const VPlan &a = P.v[i1], &b = P.v[i2];
            RowsArgs &r1 = out[i1].ra;
            const RowsArgs &r2 = out[i2].ra;
            if (!out[i1].rows || !out[i2].fused || a.MO != 1 || a.R != b.R || b.fused_from != i1)
                return fail(g, PASE_ERR_INTERNAL, "fused minimum plan");
            const void *Tp = ws + P.off_T + a.T_off;
            int own = 0;
            r1.fz_na = 0;
            for (uint32_t t = 0; t < r2.na; t++) {
                if (r2.a[t].ptr == Tp) {
                    // the reader's lookup of T_i1 must address it as the producer
                    // writes it: [z][r], z stride MR, row strides those of T_i1
                    bool same = r2.a[t].sc == a.MR;
                    for (size_t k = 0; k < a.R.size(); k++) same &= r2.a[t].sdR[k] == a.stride[1 + k];
                    if (!same) return fail(g, PASE_ERR_INTERNAL, "fused minimum lookup layout");
                    own++;
                    continue;
                }
                r1.fz_a[r1.fz_na++] = r2.a[t];
            }
            if (own != 1) return fail(g, PASE_ERR_INTERNAL, "fused minimum lookup");
            r1.fz_keys = ws + P.off_fused + b.fkeys_off;
            r1.fz_B = r2.B;
            r1.fz_ldz = r2.ldz;
            if (r1.Kz != b.K || r2.MR != a.MR) return fail(g, PASE_ERR_INTERNAL, "fused minimum shape");
            // nothing else reads T_i1 unless the tables are kept for queries
            if (!g->keep_tables) r1.T = nullptr;
        }
    }
    return PASE_OK;
}


template pase_status build_launches<double>(pase_graph_t, char *, std::vector<Launch<double>> &,
                                            std::vector<Contrib> &);
template pase_status build_launches<uint64_t>(pase_graph_t, char *, std::vector<Launch<uint64_t>> &,
                                              std::vector<Contrib> &);
template pase_status build_launches<unsigned __int128>(pase_graph_t, char *,
                                                       std::vector<Launch<unsigned __int128>> &,
                                                       std::vector<Contrib> &);

// ------------------------------------------------------------------ constant image and batches
template <typename KeyT>
pase_status build_image(pase_graph_t g, char *ws, char *img, SearchImage &si, bool allow_streams) {
    const Plan &P = g->plan;
    const int n = (int)P.v.size();
    const size_t nv = g->V.size(), ne = g->E.size();
    std::vector<Launch<KeyT>> launches;
    std::vector<Contrib> contrib;
    pase_status st = build_launches<KeyT>(g, ws, launches, contrib);
    if (st != PASE_OK) return st;
    si = SearchImage();
    si.lanes = allow_streams && P.resident && (g->schedule == kSchedBulk || g->schedule == kSchedSplit);
    si.hoist = allow_streams && !si.lanes && P.hoisted > 0;
    si.lane_hoist = si.lanes && P.hoisted > 0;
    // every piece of the image is checked against the end of its region first
    auto region = [&](uint64_t off, uint64_t bytes, uint64_t end, const char *what) {
        return off + bytes <= end && end <= P.off_cfg ? PASE_OK
                                                     : fail(g, PASE_ERR_INTERNAL, std::string("image region: ") + what);
    };

    // the layer costs, their device bytes and the split signatures
    // [off_L, off_ovedge) are written by k_cost_tables on the device: unless
    // the caller overrode the costs, that range is not cleared here, and it is
    // left out of the upload once it is large enough to pay for a second copy
    // call (what the one copy then carries there is overwritten on the device)
    si.upload_costs = g->overridden || P.off_ovedge - P.off_L < (256u << 10);
    if (g->overridden) {
        std::memset(img, 0, P.off_cfg);
    } else {
        std::memset(img, 0, P.off_L);
        std::memset(img + P.off_ovedge, 0, P.off_cfg - P.off_ovedge);
    }
    // one row set per dimension count, shared by the vertices with that count
    uint64_t row_off[kMaxDims + 1] = {0}, off = 0;
    for (size_t d = 0; d < g->ex_rows.size() && d <= (size_t)kMaxDims; d++) {
        row_off[d] = off;
        if (!g->ex_rows[d].empty()) {
            if ((st = region(P.off_ex + off, g->ex_rows[d].size(), P.off_vert, "split rows")) != PASE_OK) return st;
            std::memcpy(img + P.off_ex + off, g->ex_rows[d].data(), g->ex_rows[d].size());
        }
        off += g->ex_rows[d].size();
    }
    std::vector<DevVertex> dvs(nv);
    uint64_t loff = 0;
    for (size_t v = 0; v < nv; v++) {
        DevVertex &x = dvs[v];
        std::memset(&x, 0, sizeof x);
        x.ex_off = row_off[g->V[v].ndims];
        x.L_off = loff;
        x.flops = g->flops[v];
        x.keep_n = g->keep_n[v];
        x.K = g->K[v];
        x.ndims = g->V[v].ndims;
        x.reduce_mask = g->V[v].reduce_mask;
        x.factors = g->factors ? 1 : 0;
        x.weight_n = g->weight_n[v];
        x.weight_mask = g->V[v].weight_mask;
        if (g->halo) {
            x.input_mask = g->V[v].input_mask;
            for (uint32_t k = 0; k < kMaxDims; k++) {
                x.halo_w[k] = g->V[v].halo[k];
                x.halo_n[k] = g->halo_n[v][k];
                if (x.halo_w[k]) x.halo_mask |= 1u << k;
            }
        }
        loff += g->K[v];
    }
    si.nL = loff;
    if ((st = region(P.off_vert, nv * sizeof(DevVertex), P.off_edge, "vertices")) != PASE_OK) return st;
    std::memcpy(img + P.off_vert, dvs.data(), nv * sizeof(DevVertex));
    std::vector<DevEdge> des(ne);
    uint64_t sig_off = 0;
    for (size_t e = 0; e < ne; e++) {
        DevEdge &x = des[e];
        std::memset(&x, 0, sizeof x);
        x.src = g->E[e].src;
        x.dst = g->E[e].dst;
        x.rank = g->E[e].rank;
        x.factors = g->factors ? 1 : 0;
        for (uint32_t k = 0; k < kMaxDims; k++) {
            x.sdim[k] = (int8_t)(k < x.rank ? g->E[e].src_dim[k] : -1);
            x.ddim[k] = (int8_t)(k < x.rank ? g->E[e].dst_dim[k] : -1);
        }
        x.elems = g->E[e].elems;
        x.sig_off = sig_off;
        x.mat_off = g->volume ? g->mat_off[e] : 0;
        x.row0 = g->volume ? g->mat_row0[e] : 0;
        sig_off += (uint64_t)g->K[x.src] + g->K[x.dst];
    }
    if (ne) {
        if ((st = region(P.off_edge, ne * sizeof(DevEdge), P.off_L, "edges")) != PASE_OK) return st;
        std::memcpy(img + P.off_edge, des.data(), ne * sizeof(DevEdge));
    }
    if (g->overridden) {
        if ((st = region(P.off_L, g->ov_layer.size() * 8, P.off_lsum, "layer costs")) != PASE_OK) return st;
        std::memcpy(img + P.off_L, g->ov_layer.data(), g->ov_layer.size() * 8);
        if (!g->ov_edge.empty()) {
            if ((st = region(P.off_ovedge, g->ov_edge.size() * 8, P.off_contrib, "edge costs")) != PASE_OK) return st;
            std::memcpy(img + P.off_ovedge, g->ov_edge.data(), g->ov_edge.size() * 8);
        }
    }
    if ((st = region(P.off_contrib, contrib.size() * sizeof(Contrib), P.off_bt, "contributions")) != PASE_OK) return st;
    if (!contrib.empty()) std::memcpy(img + P.off_contrib, contrib.data(), contrib.size() * sizeof(Contrib));
    std::vector<BacktrackDesc> bt(n);
    uint32_t nlev = 0;
    for (int i = n - 1; i >= 0; i--) {
        const VPlan &vp = P.v[i];
        BacktrackDesc &b = bt[i];
        std::memset(&b, 0, sizeof b);
        b.A = (const uint16_t *)(ws + P.off_A + vp.A_off);
        b.vi = (uint32_t)vp.vi;
        b.K = vp.K;
        b.m = (uint32_t)vp.layout.size();
        for (size_t k = 0; k < vp.layout.size(); k++) {
            b.dig[k] = (uint32_t)vp.layout[k];
            b.stride[k] = vp.stride[k];
        }
        // the configuration of v_i needs those of D(i), all later in the order
        for (int u : vp.D) b.level = std::max(b.level, bt[P.pos[u]].level + 1);
        nlev = std::max(nlev, b.level + 1);
    }
    si.nlev = nlev;
    if ((st = region(P.off_bt, n * sizeof(BacktrackDesc), P.off_desc, "back-substitution")) != PASE_OK) return st;
    std::memcpy(img + P.off_bt, bt.data(), n * sizeof(BacktrackDesc));

    // ---- kernel descriptors: per position, one of each kind
    const uint64_t desc_bytes =
        (uint64_t)n * (sizeof(PrepArgs) + sizeof(RowsArgs) + sizeof(GenericArgs) + sizeof(ReduceArgs) + sizeof(DirectArgs));
    if ((st = region(P.off_desc, desc_bytes, P.off_batch, "descriptors")) != PASE_OK) return st;
    PrepArgs *hp = (PrepArgs *)(img + P.off_desc);
    RowsArgs *hr = (RowsArgs *)(hp + n);
    GenericArgs *hg = (GenericArgs *)(hr + n);
    ReduceArgs *hd = (ReduceArgs *)(hg + n);
    DirectArgs *hx = (DirectArgs *)(hd + n);
    for (int i = 0; i < n; i++) {
        hp[i] = launches[i].prep;
        hr[i] = launches[i].ra;
        hg[i] = launches[i].ga;
        hd[i] = launches[i].red;
        hx[i] = launches[i].da;
    }

    // ---- batches: per launch group, one prep launch, one fill launch per
    // kernel variant and one split-reduction launch
    BatchEntry *hbe = (BatchEntry *)(img + P.off_batch);
    const uint64_t be_cap = (P.off_zero - P.off_batch) / sizeof(BatchEntry);
    uint32_t nbe = 0;
    // launch groups in enqueue order: the slots (levels, or positions); with
    // lanes, each slot's vertices of lane 0, then those of lane 1
    const int nl = si.lanes ? kLanes : 1;
    si.groups.assign((size_t)P.nslots * nl, {});
    si.group_lane.assign(si.groups.size(), 0);
    for (int i = 0; i < n; i++) si.groups[(size_t)P.v[i].slot * nl + (si.lanes ? P.v[i].lane : 0)].push_back(i);
    for (size_t k = 0; k < si.groups.size(); k++) si.group_lane[k] = (int)(k % nl);
    int cur_lane = 0, cur_group = 0;
    bool be_overflow = false;
    auto add_batch = [&](Batch::Kind kind, uint32_t variant, const std::vector<int> &members,
                         uint32_t (*nblk)(const Launch<KeyT> &)) {
        if (members.empty()) return;
        Batch b{kind, cur_lane, cur_group, variant, nbe, 0, 0, false};
        for (int i : members) {
            if (nbe >= be_cap) { be_overflow = true; return; }
            hbe[nbe].pos = (uint32_t)i;
            hbe[nbe].first = b.blocks;
            hbe[nbe].prio = si.lanes && P.v[i].lane == 0 ? 1u : 0u;
            hbe[nbe].kind = 0;
            b.blocks += nblk(launches[i]);
            nbe++;
            b.nentries++;
        }
        si.batches.push_back(b);
    };
    // per-group scratch, reused across groups (cleared, capacity kept)
    std::vector<int> prepped, direct, grp;
    std::vector<std::pair<uint32_t, int>> rows, gens, reds;
    std::map<uint32_t, int> shape_dom;   // TZ * 4 + TM -> largest vertex of the group
    constexpr bool kF64 = std::is_same<KeyT, double>::value;
    // hoisted preps: a side batch after the group of the slot whose tables
    // they read last (before group 0 when they read none); each vertex's group
    // waits for its side batch
    std::vector<std::vector<int>> hoist_after(si.groups.size() + 1);   // [slot + 1] -> positions
    si.group_waits.assign(si.groups.size(), {});
    if (si.hoist)
        for (int i = 0; i < n; i++)
            if (P.v[i].prep_after >= -1) hoist_after[(size_t)(P.v[i].prep_after + 1)].push_back(i);
    // with lanes: a hoisted prep is a prep batch of its own at the end of the
    // group (prep_after, lane of the tables it reads)
    std::vector<std::vector<int>> lane_hoist_at(si.groups.size());   // group -> positions
    if (si.lane_hoist)
        for (int i = 0; i < n; i++)
            if (P.v[i].prep_after >= 0)
                lane_hoist_at[(size_t)P.v[i].prep_after * nl + P.v[i].prep_lane].push_back(i);
    const bool hoisting = si.hoist || si.lane_hoist;
    auto add_side = [&](size_t k) {
        if (hoist_after[k].empty()) return;
        const int bi = (int)si.batches.size();
        add_batch(Batch::kPrep, 0, hoist_after[k], [](const Launch<KeyT> &L) { return L.prep.nwg; });
        if ((int)si.batches.size() == bi + 1) si.batches.back().side = true;
        for (int i : hoist_after[k]) si.group_waits[(size_t)P.v[i].slot].push_back(bi);
    };
    add_side(0);
    for (size_t sl = 0; sl < si.groups.size(); sl++) {
        const auto &mem = si.groups[sl];
        cur_lane = si.group_lane[sl];
        cur_group = (int)sl;
        prepped.clear();
        direct.clear();
        // a fused minimum's blocks are built with its producer's, before the
        // producer's fill reads them; its own fill is a reduction (below)
        std::vector<int> fills;   // members with a prep here or hoisted: rows / generic fills
        for (int i : mem) {
            if (launches[i].direct) direct.push_back(i);
            else if (!launches[i].fused) (hoisting && P.v[i].prep_after >= -1 ? fills : prepped).push_back(i);
            if (P.v[i].fuse_into >= 0) prepped.push_back(P.v[i].fuse_into);
        }
        add_batch(Batch::kDirect, 0, direct, [](const Launch<KeyT> &L) { return L.da.nblk; });
        add_batch(Batch::kPrep, 0, prepped, [](const Launch<KeyT> &L) { return L.prep.nwg; });
        prepped.insert(prepped.end(), fills.begin(), fills.end());
        rows.clear();
        gens.clear();
        reds.clear();
        // fp64 keys: the row-term count is a kernel template parameter; a
        // small vertex with fewer row terms than the largest vertex of its tile
        // shape in this group gets zero terms appended (each lane adds the
        // zero key once per c) and joins that vertex's launch
        shape_dom.clear();
        for (int i : prepped)
            if (launches[i].rows && !launches[i].fused && kF64) {
                auto it = shape_dom.find(P.v[i].TZ * 4 + P.v[i].TM);
                if (it == shape_dom.end()) shape_dom[P.v[i].TZ * 4 + P.v[i].TM] = i;
                else if (P.v[i].est_us > P.v[it->second].est_us) it->second = i;
            }
        for (int i : prepped) {
            const Launch<KeyT> &L = launches[i];
            if (L.fused) continue;
            if (L.rows) {
                uint32_t na = kF64 ? std::min<uint32_t>(L.ra.na, 4) : 7;
                if (kF64) {
                    const int d = shape_dom[P.v[i].TZ * 4 + P.v[i].TM];
                    const uint32_t nd = std::min<uint32_t>(launches[d].ra.na, 4);
                    if (d != i && na < nd && P.v[i].est_us <= 0.5 * P.v[d].est_us) {
                        RowsArgs &ra = hr[i];
                        for (uint32_t t = na; t < nd; t++) {
                            std::memset(&ra.a[t], 0, sizeof ra.a[t]);
                            ra.a[t].ptr = ws + P.off_zero;
                            ra.a[t].bytes = 8;
                        }
                        na = nd;
                    }
                }
                rows.push_back({(P.v[i].TZ * 4 + P.v[i].TM) * 8 + na, i});
                if (P.v[i].nsplit > 1) reds.push_back({0, i});
            } else {
                gens.push_back({L.ga.nt <= 6 ? L.ga.nt : 0, i});
            }
        }
        auto by_variant = [](const std::pair<uint32_t, int> &a, const std::pair<uint32_t, int> &b) {
            return a.first < b.first;
        };
        std::stable_sort(rows.begin(), rows.end(), by_variant);
        std::stable_sort(gens.begin(), gens.end(), by_variant);
        // two-term generic fills of the group ride along in its largest row
        // launch (64-bit keys) instead of a generic launch of their own
        std::vector<int> ride;
        uint32_t ride_variant = ~0u;
        if constexpr (sizeof(KeyT) == 8) {
            uint64_t best = 0;
            for (size_t k = 0; k < rows.size();) {
                size_t k2 = k;
                uint64_t blocks = 0;
                for (; k2 < rows.size() && rows[k2].first == rows[k].first; k2++)
                    blocks += launches[rows[k2].second].ra.nblocks_launched;
                if (ride_variant == ~0u || blocks > best) { best = blocks; ride_variant = rows[k].first; }
                k = k2;
            }
            if (ride_variant != ~0u) {
                std::vector<std::pair<uint32_t, int>> keep;
                for (const auto &x : gens) {
                    if (launches[x.second].ga.nt == 2) ride.push_back(x.second);
                    else keep.push_back(x);
                }
                gens.swap(keep);
            }
        }
        for (size_t k = 0; k < rows.size();) {
            grp.clear();
            size_t k2 = k;
            for (; k2 < rows.size() && rows[k2].first == rows[k].first; k2++) grp.push_back(rows[k2].second);
            add_batch(Batch::kRows, rows[k].first, grp, [](const Launch<KeyT> &L) { return L.ra.nblocks_launched; });
            if (rows[k].first == ride_variant && !si.batches.empty()) {
                Batch &b = si.batches.back();
                for (int i : ride) {
                    if (nbe >= be_cap) { be_overflow = true; break; }
                    hbe[nbe].pos = (uint32_t)i;
                    hbe[nbe].first = b.blocks;
                    hbe[nbe].prio = si.lanes && P.v[i].lane == 0 ? 1u : 0u;
                    hbe[nbe].kind = kEntryGeneric2;
                    b.blocks += launches[i].ga.nblk;
                    nbe++;
                    b.nentries++;
                }
            }
            k = k2;
        }
        for (size_t k = 0; k < gens.size();) {
            grp.clear();
            size_t k2 = k;
            for (; k2 < gens.size() && gens[k2].first == gens[k].first; k2++) grp.push_back(gens[k2].second);
            add_batch(Batch::kGeneric, gens[k].first, grp, [](const Launch<KeyT> &L) { return L.ga.nblk; });
            k = k2;
        }
        for (int i : mem)
            if (launches[i].fused) reds.push_back({0, i});
        grp.clear();
        for (auto &x : reds) grp.push_back(x.second);
        add_batch(Batch::kReduce, 0, grp, [](const Launch<KeyT> &L) { return L.red.nblk; });
        add_batch(Batch::kPrep, 0, lane_hoist_at[sl], [](const Launch<KeyT> &L) { return L.prep.nwg; });
        if (be_overflow) return fail(g, PASE_ERR_INTERNAL, "batch table overflow");
        add_side(sl + 1);
    }
    for (const Batch &b : si.batches)
        if (b.blocks == 0 || b.blocks > 0x7fffffffu) return fail(g, PASE_ERR_TOO_LARGE, "launch grid size");
    return PASE_OK;
}

template pase_status build_image<double>(pase_graph_t, char *, char *, SearchImage &, bool);
template pase_status build_image<uint64_t>(pase_graph_t, char *, char *, SearchImage &, bool);
template pase_status build_image<unsigned __int128>(pase_graph_t, char *, char *, SearchImage &, bool);

pase_status plan_check(pase_graph_t g, uint64_t *image_bytes) {
    // descriptors only hold device addresses: any base will do, nothing is
    // read through it; the image buffer is exactly the constant region, so a
    // write past it is a heap overflow (and a sanitizer build reports it)
    char *fake_ws = (char *)(uintptr_t)(1ull << 40);
    const uint64_t bytes = g->plan.off_cfg;
    std::vector<char> img(bytes);
    SearchImage si;
    pase_status st = g->plan_key_type == 0   ? build_image<double>(g, fake_ws, img.data(), si)
                     : g->plan_key_type == 1 ? build_image<uint64_t>(g, fake_ws, img.data(), si)
                                             : build_image<unsigned __int128>(g, fake_ws, img.data(), si);
    if (st != PASE_OK) return st;
    // every vertex appears in exactly one fill batch (direct, row or generic)
    std::vector<int> fills(g->plan.v.size(), 0);
    const BatchEntry *be = (const BatchEntry *)(img.data() + g->plan.off_batch);
    std::vector<int> prep_batch(g->plan.v.size(), -1), fill_batch(g->plan.v.size(), -1);
    for (size_t bi = 0; bi < si.batches.size(); bi++) {
        const Batch &b = si.batches[bi];
        for (uint32_t k = 0; k < b.nentries; k++) {
            const uint32_t pos = be[b.entry0 + k].pos;
            if (pos >= fills.size()) return fail(g, PASE_ERR_INTERNAL, "batch entry out of range");
            const bool fused = g->plan.v[pos].fused_from >= 0;
            if (b.kind == Batch::kRows || b.kind == Batch::kGeneric || b.kind == Batch::kDirect ||
                (b.kind == Batch::kReduce && fused)) {
                fills[pos]++;
                fill_batch[pos] = (int)bi;
            }
            if (b.kind == Batch::kPrep) prep_batch[pos] = (int)bi;
        }
    }
    // every vertex with blocks has them built before its fill; a hoisted
    // prep's side batch comes after the fills of the slot it waits for and is
    // waited for by the vertex's group
    for (size_t i = 0; i < g->plan.v.size(); i++) {
        const VPlan &vp = g->plan.v[i];
        if (vp.kernel == kDirect || vp.fused_from >= 0) continue;
        if (prep_batch[i] < 0 || prep_batch[i] > fill_batch[i])
            return fail(g, PASE_ERR_INTERNAL, "a prep does not precede its fill");
        if (si.hoist && vp.prep_after >= -1) {
            const Batch &b = si.batches[prep_batch[i]];
            const auto &w = si.group_waits[(size_t)vp.slot];
            if (!b.side || std::find(w.begin(), w.end(), prep_batch[i]) == w.end())
                return fail(g, PASE_ERR_INTERNAL, "a hoisted prep is not waited for");
            for (size_t k = 0; k < (size_t)prep_batch[i]; k++)
                if (si.batches[k].group > vp.prep_after && !si.batches[k].side)
                    return fail(g, PASE_ERR_INTERNAL, "a hoisted prep runs after a later slot");
            for (size_t k = prep_batch[i] + 1; k < si.batches.size(); k++)
                if (si.batches[k].group <= vp.prep_after && !si.batches[k].side)
                    return fail(g, PASE_ERR_INTERNAL, "a hoisted prep runs before the tables it reads");
        }
        // with lanes: at the end of group (prep_after, prep_lane), after the
        // fills of that lane's tables up to that slot (the ones its blocks
        // read among them); on another lane than the vertex's, the vertex
        // reads a table of the prep's lane at that slot or later, so its group
        // waits for that lane past the prep
        if (si.lane_hoist && vp.prep_after >= 0) {
            const Batch &b = si.batches[prep_batch[i]];
            if (b.lane != vp.prep_lane || b.group != vp.prep_after * kLanes + vp.prep_lane)
                return fail(g, PASE_ERR_INTERNAL, "a hoisted prep is not on its lane");
            bool waited = vp.prep_lane == vp.lane;
            for (const auto &t : vp.terms) {
                const VPlan &pj = g->plan.v[t.j];
                if (pj.slot <= vp.prep_after && pj.lane == vp.prep_lane && fill_batch[t.j] > prep_batch[i])
                    return fail(g, PASE_ERR_INTERNAL, "a hoisted prep runs before the tables it reads");
                waited |= pj.lane == vp.prep_lane && pj.slot >= vp.prep_after;
            }
            if (!waited) return fail(g, PASE_ERR_INTERNAL, "a hoisted prep on another lane is not waited for");
        }
    }
    // a fused minimum: its blocks are built before its producer's fill, and its
    // reduction comes after that fill
    for (size_t i = 0; i < g->plan.v.size(); i++) {
        const int j = g->plan.v[i].fused_from;
        if (j < 0) continue;
        if (prep_batch[i] < 0 || fill_batch[j] < 0 || prep_batch[i] > fill_batch[j] || fill_batch[i] < fill_batch[j])
            return fail(g, PASE_ERR_INTERNAL, "fused minimum out of order");
    }
    for (int f : fills)
        if (f != 1) return fail(g, PASE_ERR_INTERNAL, "a vertex is not filled exactly once");
    *image_bytes = bytes;
    return PASE_OK;
}

}  // namespace pase
