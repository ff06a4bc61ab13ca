// Device runtime and HIP kernels of libpase (gfx950).
//
// FindBestStrategy (Fig. 4) runs as: one cost-table kernel for all layer
// costs; then, for each position i of the GenerateSeq order, a prep kernel
// that folds every term of recurrence (4) depending on at most (c, one digit)
// -- or, for the row kernel, on (c, outer digits, column digit) -- into
// key-space blocks, and one fill kernel that evaluates
//     T_i[phi] = min_c  sum of terms(phi, c)      (and the minimising c)
// for every phi; finally one back-substitution kernel.
//
// Keys.  A key is cost * 2^b + c with b = ceil(log2 K_i): the minimum key
// gives the minimum cost and, among equal costs, the lowest configuration
// index -- exactly the strict "<" update of Fig. 4 over ascending indices.
// When the host proves every key is below 2^53 (sum of the maximal layer and
// transfer costs, shifted by b), keys are doubles: every add of two keys is
// then exact integer arithmetic and min-plus costs one v_add_f64 and one
// v_min_f64 per cell.  Otherwise keys are uint64.
#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>

#include <algorithm>
#include <chrono>
#include <map>
#include <type_traits>
#include <cstring>
#include <numeric>
#include <vector>

#include "internal.h"
#include "kernels.h"

using namespace pase;

// Cost tables of the search: layer cost and device byte (device count or its
// log2) of every (vertex, configuration), and the split signatures of every
// (edge endpoint, configuration); r * t_x(e, cu, cv) is then read off two
// signatures and two device bytes (edge_cost_sig).
__global__ void k_cost_tables(const DevVertex *__restrict__ V, uint32_t nv, const DevEdge *__restrict__ E,
                              uint32_t ne, const uint8_t *__restrict__ ex, uint64_t *__restrict__ L,
                              uint8_t *__restrict__ lsum, uint64_t *__restrict__ sig, uint64_t nL,
                              uint64_t nS, uint64_t r) {
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < nL + nS;
         t += (uint64_t)gridDim.x * blockDim.x) {
        if (t < nL) {
            uint32_t lo = 0, hi = nv;   // last vertex with L_off <= t
            while (hi - lo > 1) {
                uint32_t mid = (lo + hi) / 2;
                if (V[mid].L_off <= t) lo = mid; else hi = mid;
            }
            const DevVertex dv = V[lo];
            const uint8_t *e = ex + dv.ex_off + (t - dv.L_off) * dv.ndims;
            L[t] = layer_cost(dv, e, r);
            lsum[t] = (uint8_t)device_byte(dv, e);
        } else {
            uint64_t u = t - nL;
            uint32_t lo = 0, hi = ne;   // last edge with sig_off <= u
            while (hi - lo > 1) {
                uint32_t mid = (lo + hi) / 2;
                if (E[mid].sig_off <= u) lo = mid; else hi = mid;
            }
            const DevEdge de = E[lo];
            uint64_t c = u - de.sig_off;
            const DevVertex vs = V[de.src];
            if (c < vs.K) {
                sig[u] = split_signature(de.sdim, de.rank, ex + vs.ex_off + c * vs.ndims, de.factors);
            } else {
                const DevVertex vd = V[de.dst];
                c -= vs.K;
                sig[u] = split_signature(de.ddim, de.rank, ex + vd.ex_off + c * vd.ndims, de.factors);
            }
        }
    }
}

// Volume-intersection model: every entry of every edge's K_src x K_dst cost
// matrix (one thread per entry, grid-stride), into the matrix region the prep
// kernel then reads like caller-given matrices.
__global__ void k_edge_volume(const DevVertex *__restrict__ V, const DevEdge *__restrict__ E, uint32_t ne,
                              const uint8_t *__restrict__ ex, uint64_t *__restrict__ out, uint64_t total,
                              uint64_t r) {
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < total;
         t += (uint64_t)gridDim.x * blockDim.x) {
        uint32_t lo = 0, hi = ne;   // last edge with mat_off <= t
        while (hi - lo > 1) {
            uint32_t mid = (lo + hi) / 2;
            if (E[mid].mat_off <= t) lo = mid; else hi = mid;
        }
        const DevEdge de = E[lo];
        const DevVertex u = V[de.src], v = V[de.dst];
        const uint64_t x = t - de.mat_off, cu = x / v.K, cv = x % v.K;
        out[t] = volume_cost(u, ex + u.ex_off + cu * u.ndims, v, ex + v.ex_off + cv * v.ndims, de, r);
    }
}

__global__ void k_edge_costs(const DevVertex *__restrict__ V, const DevEdge *__restrict__ E, uint32_t e,
                             const uint8_t *__restrict__ lsum, const uint64_t *__restrict__ sig,
                             uint64_t *__restrict__ out, uint64_t r) {
    const DevEdge de = E[e];
    const DevVertex u = V[de.src], v = V[de.dst];
    uint64_t total = (uint64_t)u.K * v.K;
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < total;
         t += (uint64_t)gridDim.x * blockDim.x) {
        uint64_t cu = t / v.K, cv = t % v.K;
        out[t] = edge_cost_sig(sig[de.sig_off + cu], sig[de.sig_off + u.K + cv], lsum[u.L_off + cu],
                               lsum[v.L_off + cv], de.elems, r, de.factors);
    }
}

template <typename KeyT>
__global__ __launch_bounds__(kPrepThreads) void k_prep(const PrepArgs *__restrict__ descs,
                                                     const BatchEntry *__restrict__ be, uint32_t nbe,
                                                     const DevVertex *__restrict__ V,
                                                     const DevEdge *__restrict__ E,
                                                     const uint64_t *__restrict__ L,
                                                     const uint8_t *__restrict__ lsum,
                                                     const uint64_t *__restrict__ sig,
                                                     const Contrib *__restrict__ cb, uint64_t r) {
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    set_priority(be[kb]);
    prep_item<KeyT>(descs[be[kb].pos], blockIdx.x - be[kb].first, V, E, L, lsum, sig, cb, r);
}

template <typename KeyT, int TZ, int TM, int NA>
__global__ __launch_bounds__(256) void k_fill_rows(const RowsArgs *__restrict__ descs,
                                                  const BatchEntry *__restrict__ be, uint32_t nbe) {
    __shared__ MergeBuf<KeyT> xch;
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    set_priority(be[kb]);
    rows_item<KeyT, TZ, TM, NA>(descs[be[kb].pos], blockIdx.x - be[kb].first, xch);
}

template <typename KeyT>
__global__ __launch_bounds__(256) void k_reduce_splits(const ReduceArgs *__restrict__ descs,
                                                      const BatchEntry *__restrict__ be, uint32_t nbe) {
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    set_priority(be[kb]);
    reduce_item<KeyT>(descs[be[kb].pos], blockIdx.x - be[kb].first);
}

template <typename KeyT, int NT>
__global__ __launch_bounds__(256) void k_fill_generic(const GenericArgs *__restrict__ descs,
                                                     const BatchEntry *__restrict__ be, uint32_t nbe) {
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    set_priority(be[kb]);
    generic_item<KeyT, NT>(descs[be[kb].pos], blockIdx.x - be[kb].first);
}

// Direct fill of the small vertices of one level (batched like the others).
template <typename KeyT>
__global__ __launch_bounds__(256) void k_fill_direct(const DirectArgs *__restrict__ descs,
                                                    const BatchEntry *__restrict__ be, uint32_t nbe,
                                                    const DevVertex *__restrict__ V, const DevEdge *__restrict__ E,
                                                    const uint64_t *__restrict__ L, const uint8_t *__restrict__ lsum,
                                                    const uint64_t *__restrict__ sig, const Contrib *__restrict__ cb,
                                                    uint64_t r) {
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    set_priority(be[kb]);
    direct_item<KeyT>(descs[be[kb].pos], blockIdx.x - be[kb].first, V, E, L, lsum, sig, cb, r);
}

// ------------------------------------------------------------------ back-substitution
// From the last position down: the configuration of v_i is A_i at the
// already-chosen configurations of D(i) (every member of D(i) is later in the
// sequence).  Single thread; n dependent reads.
template <typename KeyT>
__global__ void k_backtrack(const BacktrackDesc *__restrict__ bt, uint32_t n, const void *Tlast,
                            uint32_t *__restrict__ cfg, SearchOut *out, const uint32_t *flow_error) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    uint32_t status = 0;
    for (int i = (int)n - 1; i >= 0; i--) {
        const BacktrackDesc d = bt[i];
        uint64_t idx = 0;
        for (uint32_t k = 0; k < d.m; k++) idx += (uint64_t)cfg[d.dig[k]] * d.stride[k];
        uint32_t c = d.A[idx];
        // every index above is in range as long as each stored argmin is
        if (c >= d.K) { status |= 4u; c = 0; }
        cfg[d.vi] = c;
    }
    out->min_cost = KeyOps<KeyT>::val_to_u64(((const typename KeyOps<KeyT>::Val *)Tlast)[0]);
    out->status = status | (flow_error ? *flow_error : 0u);
}

// Back-substitution by backward levels: one thread per position; the
// configurations of one level depend only on those of lower levels, so a level
// costs one dependent argmin read instead of one per vertex.  Configurations
// live in LDS until the end.
template <typename KeyT>
__global__ __launch_bounds__(kMaxBacktrackThreads) void k_backtrack_levels(const BacktrackDesc *__restrict__ bt,
                                                                          uint32_t n, uint32_t nlev,
                                                                          const void *Tlast,
                                                                          uint32_t *__restrict__ cfg,
                                                                          SearchOut *out,
                                                                          const uint32_t *flow_error) {
    __shared__ uint32_t scfg[kMaxBacktrackThreads];
    __shared__ uint32_t sbad;
    const uint32_t t = threadIdx.x;
    const bool mine = t < n;
    if (t == 0) sbad = 0;
    BacktrackDesc d;
    if (mine) d = bt[t];
    __syncthreads();
    for (uint32_t lev = 0; lev < nlev; lev++) {
        if (mine && d.level == lev) {
            uint64_t idx = 0;
            for (uint32_t k = 0; k < d.m; k++) idx += (uint64_t)scfg[d.dig[k]] * d.stride[k];
            uint32_t c = d.A[idx];
            // every index above is in range as long as each stored argmin is
            if (c >= d.K) { atomicOr(&sbad, 4u); c = 0; }
            scfg[d.vi] = c;
        }
        __syncthreads();
    }
    if (mine) cfg[t] = scfg[t];
    if (t == 0) {
        out->min_cost = KeyOps<KeyT>::val_to_u64(((const typename KeyOps<KeyT>::Val *)Tlast)[0]);
        out->status = sbad | (flow_error ? *flow_error : 0u);
    }
}

// ------------------------------------------------------------------ fingerprints (tests)
struct FingerArgs {
    const void *T;
    const uint16_t *A;
    uint64_t N;
    uint32_t m, out_shift;
    uint32_t rad[kMaxDep];
    uint64_t cstride[kMaxDep];
    unsigned long long *out;
};

__device__ __forceinline__ uint64_t splitmix64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

template <typename KeyT>
__global__ void k_fingerprint(FingerArgs a) {
    using Val = typename KeyOps<KeyT>::Val;
    uint64_t st = 0, sa = 0;
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < a.N;
         t += (uint64_t)gridDim.x * blockDim.x) {
        uint64_t x = t, canon = 0;
        for (int k = (int)a.m - 1; k >= 0; k--) {
            canon += (x % a.rad[k]) * a.cstride[k];
            x /= a.rad[k];
        }
        uint64_t h = splitmix64_mix(canon);
        st += splitmix64_mix(h ^ (KeyOps<KeyT>::val_to_u64(((const Val *)a.T)[t]) >> a.out_shift));
        sa += splitmix64_mix(h ^ (uint64_t)a.A[t]);
    }
    __shared__ uint64_t red[2][256];
    red[0][threadIdx.x] = st;
    red[1][threadIdx.x] = sa;
    __syncthreads();
    for (uint32_t s = blockDim.x / 2; s > 0; s >>= 1) {
        if (threadIdx.x < s) {
            red[0][threadIdx.x] += red[0][threadIdx.x + s];
            red[1][threadIdx.x] += red[1][threadIdx.x + s];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        atomicAdd(a.out, (unsigned long long)red[0][0]);
        atomicAdd(a.out + 1, (unsigned long long)red[1][0]);
    }
}

// ------------------------------------------------------------------ runtime
namespace pase {

constexpr int kLanes = 3;   // streams of the lane schedule

struct DeviceState {
    void *ws = nullptr;
    uint64_t ws_bytes = 0;
    bool owned = false;
    void *lent = nullptr;
    uint64_t lent_bytes = 0;
    void *pinned = nullptr;
    uint64_t pinned_bytes = 0;
    std::vector<hipEvent_t> ev;        // profiling: two per fill launch (timed)
    hipStream_t last_stream = nullptr;
    int flow_grid[2] = {0, 0};         // resident workgroups of the dataflow kernel, per key type
    int wall_khz = 0;                  // device wall clock (wall_clock64) rate
    hipStream_t side[kLanes - 1] = {}; // lane schedule: the streams of lanes 1.. (default priority)
    std::vector<hipEvent_t> lane_ev;   // lane schedule: joins (no timing)
};

#define HIPCHK(x)                                                                              \
    do {                                                                                       \
        hipError_t e_ = (x);                                                                   \
        if (e_ != hipSuccess)                                                                  \
            return fail(g, PASE_ERR_HIP, std::string(#x) + ": " + hipGetErrorString(e_));      \
    } while (0)

void device_release(pase_graph_t g) {
    DeviceState *d = g->dev;
    if (!d) return;
    if (d->owned && d->ws) (void)hipFree(d->ws);
    if (d->pinned) (void)hipHostFree(d->pinned);
    for (auto e : d->ev) (void)hipEventDestroy(e);
    for (auto e : d->lane_ev) (void)hipEventDestroy(e);
    for (auto st : d->side)
        if (st) (void)hipStreamDestroy(st);
    delete d;
    g->dev = nullptr;
}

static DeviceState *state(pase_graph_t g) {
    if (!g->dev) g->dev = new DeviceState();
    return g->dev;
}

pase_status device_set_workspace(pase_graph_t g, void *ptr, uint64_t bytes) {
    DeviceState *d = state(g);
    d->lent = ptr;
    d->lent_bytes = ptr ? bytes : 0;
    g->searched = false;
    return PASE_OK;
}

static pase_status ensure_memory(pase_graph_t g, char **ws) {
    DeviceState *d = state(g);
    const uint64_t need = g->plan.total;
    if (d->lent) {
        if (d->lent_bytes < need)
            return fail(g, PASE_ERR_OUT_OF_MEMORY, "lent workspace smaller than pase_workspace_size");
        *ws = (char *)d->lent;
    } else {
        if (!d->owned || d->ws_bytes < need) {
            if (d->owned && d->ws) HIPCHK(hipFree(d->ws));
            d->ws = nullptr;
            d->owned = false;
            if (hipMalloc(&d->ws, need) != hipSuccess) {
                (void)hipGetLastError();
                d->ws = nullptr;
                return fail(g, PASE_ERR_OUT_OF_MEMORY, "device allocation of the workspace failed");
            }
            d->owned = true;
            d->ws_bytes = need;
        }
        *ws = (char *)d->ws;
    }
    const uint64_t pin_need = g->plan.off_cfg;
    if (d->pinned_bytes < pin_need || !d->pinned) {
        if (d->pinned) HIPCHK(hipHostFree(d->pinned));
        d->pinned = nullptr;
        HIPCHK(hipHostMalloc(&d->pinned, std::max<uint64_t>(pin_need, 4096)));
        d->pinned_bytes = std::max<uint64_t>(pin_need, 4096);
    }
    return PASE_OK;
}

static uint32_t grid_for(uint64_t n, uint32_t block = 256, uint32_t cap = 8192) {
    uint64_t b = (n + block - 1) / block;
    return (uint32_t)std::max<uint64_t>(1, std::min<uint64_t>(b, cap));
}

// One vertex's launch description, resolved against the workspace base.
template <typename KeyT>
struct Launch {
    PrepArgs prep;
    bool rows = false;
    bool direct = false;
    RowsArgs ra;
    GenericArgs ga;
    ReduceArgs red;
    DirectArgs da;
};

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
static pase_status build_launches(pase_graph_t g, char *ws, std::vector<Launch<KeyT>> &out,
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
            // lanes per entry: enough threads to fill the GPU, at most one wave, at most K
            da.group_log2 = 0;
            while (da.group_log2 < 6 && (vp.N << da.group_log2) < 65536 && (2u << da.group_log2) <= vp.K)
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
            if (vp.nsplit > 1) {
                L.red.nblk = grid_for(vp.N);
                L.red.partial = ra.partial;
                L.red.T = ra.T;
                L.red.A = ra.A;
                L.red.N = vp.N;
                L.red.nsplit = vp.nsplit;
                L.red.bits = vp.bits;
                L.red.out_shift = vp.out_shift;
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
    return PASE_OK;
}

// ------------------------------------------------------------------ dataflow segments
// Vertices whose planned fill takes at least this long (us, whole GPU) go to
// the bulk queue; the rest -- the long chains of small dependent vertices --
// to the latency queue.
constexpr double kBulkUs = 25.0;

struct FlowPlan {
    std::vector<Seg> seg[2];
    std::vector<SegDep> deps;
    uint32_t nitems[2] = {0, 0};
};

// Segments (prep, fill, split reduction of every position) in one global
// order: by the start time of their vertex in a simulation of the schedule
// (latency vertices start when their producers end; bulk vertices also wait
// for the previous bulk vertex), then position, then phase.  Every vertex
// starts strictly after its producers end, so the order is topological.
template <typename KeyT>
static pase_status build_flow(pase_graph_t g, const std::vector<Launch<KeyT>> &launches, FlowPlan &fp) {
    const Plan &P = g->plan;
    const int n = (int)P.v.size();
    std::vector<uint32_t> np(n), nf(n), nr(n);
    std::vector<char> bulk(n);
    for (int i = 0; i < n; i++) {
        const Launch<KeyT> &L = launches[i];
        np[i] = L.prep.nwg;
        nf[i] = L.rows ? L.ra.nblocks_launched : L.ga.nblk;
        nr[i] = (L.rows && P.v[i].nsplit > 1) ? L.red.nblk : 0;
        bulk[i] = P.v[i].est_us >= kBulkUs;
        if (np[i] == 0 || nf[i] == 0) return fail(g, PASE_ERR_INTERNAL, "empty segment");
    }
    const double delta = 2.0;
    std::vector<int> order(n);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return P.v[a].level < P.v[b].level; });
    std::vector<double> esi(n, 0.0), efi(n, 0.0);
    for (int i : order) {
        for (const auto &t : P.v[i].terms) esi[i] = std::max(esi[i], efi[t.j]);
        efi[i] = esi[i] + P.v[i].est_us + delta;
    }
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return esi[a] < esi[b]; });
    std::vector<double> start(n, 0.0), fin(n, 0.0);
    double bulk_free = 0;
    for (int i : order) {
        double r = 0;
        for (const auto &t : P.v[i].terms) r = std::max(r, fin[t.j]);
        start[i] = bulk[i] ? std::max(r, bulk_free) : r;
        fin[i] = start[i] + P.v[i].est_us + delta;
        if (bulk[i]) bulk_free = start[i] + P.v[i].est_us;
    }
    struct Item { double key; int pos, phase; };
    std::vector<Item> items;
    for (int i = 0; i < n; i++) {
        items.push_back({start[i], i, 0});
        items.push_back({start[i], i, 1});
        if (nr[i]) items.push_back({start[i], i, 2});
    }
    std::sort(items.begin(), items.end(), [](const Item &a, const Item &b) {
        if (a.key != b.key) return a.key < b.key;
        if (a.pos != b.pos) return a.pos < b.pos;
        return a.phase < b.phase;
    });
    // check the order before anything runs: a vertex's segments come after
    // all segments of every producer it reads, and in phase order
    std::vector<int> last_idx(n, -1), first_idx(n, -1);
    for (size_t k = 0; k < items.size(); k++) {
        const int i = items[k].pos;
        if (first_idx[i] < 0) first_idx[i] = (int)k;
        if (last_idx[i] >= 0 && items[last_idx[i]].phase >= items[k].phase)
            return fail(g, PASE_ERR_INTERNAL, "dataflow order: phases out of order");
        last_idx[i] = (int)k;
    }
    for (int i = 0; i < n; i++)
        for (const auto &t : P.v[i].terms)
            if (last_idx[t.j] >= first_idx[i]) return fail(g, PASE_ERR_INTERNAL, "dataflow order not topological");
    fp = FlowPlan();
    for (const Item &it : items) {
        const int i = it.pos;
        const int q = bulk[i] ? kBulkQ : kLatQ;
        Seg sg;
        std::memset(&sg, 0, sizeof sg);
        sg.first = fp.nitems[q];
        sg.pos = (uint32_t)i;
        sg.dep_begin = (uint32_t)fp.deps.size();
        if (it.phase == 0) {
            sg.kind = kSegPrep;
            sg.count = np[i];
            for (const auto &t : P.v[i].terms) fp.deps.push_back({(uint32_t)t.j, np[t.j] + nf[t.j] + nr[t.j]});
        } else if (it.phase == 1) {
            const Launch<KeyT> &L = launches[i];
            if (L.rows) {
                sg.kind = kSegRows;
                const uint32_t na = std::is_same<KeyT, double>::value ? std::min<uint32_t>(L.ra.na, 4) : 7;
                sg.variant = (P.v[i].TZ * 4 + P.v[i].TM) * 8 + na;
            } else {
                sg.kind = kSegGeneric;
                sg.variant = L.ga.nt <= 6 ? L.ga.nt : 0;
            }
            sg.count = nf[i];
            fp.deps.push_back({(uint32_t)i, np[i]});
        } else {
            sg.kind = kSegReduce;
            sg.count = nr[i];
            fp.deps.push_back({(uint32_t)i, np[i] + nf[i]});
        }
        sg.dep_end = (uint32_t)fp.deps.size();
        if ((uint64_t)fp.nitems[q] + sg.count > 0x7fffffffull) return fail(g, PASE_ERR_TOO_LARGE, "dataflow items");
        fp.nitems[q] += sg.count;
        fp.seg[q].push_back(sg);
    }
    return PASE_OK;
}

// Randomized simulation of the k_flow worker protocol on the host: `workers`
// workgroups, the first `lat_workers` of them latency workers, take tickets
// exactly as the kernel does, wait until the dependencies of their item are
// met, run it for a random time and count it as done.  Fails if the workers
// can no longer make progress (deadlock), if an item would start before its
// dependencies are met, or if a counter does not end at its vertex's item
// count.
static pase_status flow_simulate(pase_graph_t g, const FlowPlan &fp, uint32_t workers, uint32_t lat_workers,
                                 uint64_t seed) {
    const int n = (int)g->plan.v.size();
    std::vector<uint32_t> done(n, 0), total(n, 0);
    for (int q = 0; q < 2; q++)
        for (const Seg &sg : fp.seg[q]) total[sg.pos] += sg.count;
    auto seg_of = [&](int q, uint32_t t) -> const Seg & {
        size_t lo = 0, hi = fp.seg[q].size();
        while (hi - lo > 1) {
            const size_t mid = (lo + hi) / 2;
            if (fp.seg[q][mid].first <= t) lo = mid; else hi = mid;
        }
        return fp.seg[q][lo];
    };
    auto met = [&](const Seg &sg) {
        for (uint32_t k = sg.dep_begin; k < sg.dep_end; k++)
            if (done[fp.deps[k].counter] < fp.deps[k].target) return false;
        return true;
    };
    for (const SegDep &d : fp.deps)
        if (d.counter >= (uint32_t)n || d.target > total[d.counter])
            return fail(g, PASE_ERR_INTERNAL, "dataflow dependency can never be met");
    enum { kIdle, kWaiting, kRunning, kExited };
    struct W { bool lat; int state; int q; uint32_t t; double until; };
    std::vector<W> w(workers);
    for (uint32_t k = 0; k < workers; k++) w[k] = {k < lat_workers, kIdle, -1, 0, 0.0};
    uint64_t head[2] = {0, 0};
    uint64_t rs = seed * 0x9E3779B97F4A7C15ull + 1;
    auto rnd = [&]() {   // xorshift64*
        rs ^= rs >> 12; rs ^= rs << 25; rs ^= rs >> 27;
        return rs * 0x2545F4914F6CDD1Dull;
    };
    std::vector<uint32_t> idx(workers);
    std::iota(idx.begin(), idx.end(), 0u);
    double now = 0;
    for (;;) {
        for (uint32_t k = workers; k > 1; k--) std::swap(idx[k - 1], idx[rnd() % k]);
        for (uint32_t k : idx) {
            W &x = w[k];
            if (x.state != kIdle) continue;
            int q = -1;
            uint64_t t = 0;
            if (x.lat) {
                t = head[kLatQ]++;
                if (t < fp.nitems[kLatQ]) q = kLatQ; else x.lat = false;
            }
            if (q < 0 && head[kLatQ] < fp.nitems[kLatQ] && met(seg_of(kLatQ, (uint32_t)head[kLatQ]))) {
                t = head[kLatQ]++;
                q = kLatQ;
            }
            if (q < 0) {
                t = head[kBulkQ]++;
                if (t < fp.nitems[kBulkQ]) {
                    q = kBulkQ;
                } else {
                    t = head[kLatQ]++;
                    if (t < fp.nitems[kLatQ]) q = kLatQ;
                }
            }
            if (q < 0) { x.state = kExited; continue; }
            x.q = q;
            x.t = (uint32_t)t;
            x.state = kWaiting;
        }
        bool any_running = false, any_waiting = false;
        for (W &x : w) {
            if (x.state == kWaiting && met(seg_of(x.q, x.t))) {
                x.state = kRunning;
                x.until = now + 1.0 + (double)(rnd() % 1000) / 100.0;
            }
            any_running |= x.state == kRunning;
            any_waiting |= x.state == kWaiting;
        }
        if (!any_running) {
            if (any_waiting) return fail(g, PASE_ERR_INTERNAL, "dataflow schedule deadlocks");
            break;
        }
        double next = 1e300;
        for (const W &x : w)
            if (x.state == kRunning) next = std::min(next, x.until);
        now = next;
        for (W &x : w)
            if (x.state == kRunning && x.until <= now) {
                done[seg_of(x.q, x.t).pos]++;
                x.state = kIdle;
            }
    }
    for (int i = 0; i < n; i++)
        if (done[i] != total[i]) return fail(g, PASE_ERR_INTERNAL, "dataflow items left undone");
    return PASE_OK;
}

// A batched launch: vertices (sequence positions) sharing one kernel variant
// within one launch slot, with their first workgroups.
struct Batch {
    enum Kind { kPrep, kRows, kGeneric, kReduce, kDirect } kind;
    int lane;              // two-lane schedule: the stream it runs on
    int group;             // launch group (a slot, or a (level, lane) pair) it belongs to
    uint32_t variant;      // rows: (TZ * 4 + TM) * 8 + NA (NA 7 = runtime count); generic: NT (0 = runtime)
    uint32_t entry0;       // first BatchEntry of this batch
    uint32_t nentries;
    uint32_t blocks;       // workgroups of the launch
};

template <typename KeyT, int TZ, int TM>
static void launch_rows_tz(const RowsArgs *descs, const BatchEntry *be, const Batch &b, hipStream_t s, hipEvent_t e0,
                           hipEvent_t e1) {
    dim3 grid(b.blocks), block(256);
    const uint32_t na = b.variant % 8;
    if constexpr (std::is_same<KeyT, double>::value) {
        switch (na) {
        case 0: hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, 0>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
        case 1: hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, 1>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
        case 2: hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, 2>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
        case 3: hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, 3>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
        default: hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, 4>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
        }
    } else {
        hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, -1>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries);
    }
}

// variant = (TZ * 4 + TM) * 8 + NA
template <typename KeyT>
static bool launch_rows(const RowsArgs *descs, const BatchEntry *be, const Batch &b, hipStream_t s, hipEvent_t e0,
                        hipEvent_t e1) {
    switch (b.variant / 8) {
    case 1 * 4 + 1: launch_rows_tz<KeyT, 1, 1>(descs, be, b, s, e0, e1); return true;
    case 1 * 4 + 2: launch_rows_tz<KeyT, 1, 2>(descs, be, b, s, e0, e1); return true;
    case 8 * 4 + 1: launch_rows_tz<KeyT, 8, 1>(descs, be, b, s, e0, e1); return true;
    case 8 * 4 + 2: launch_rows_tz<KeyT, 8, 2>(descs, be, b, s, e0, e1); return true;
    case 12 * 4 + 1: launch_rows_tz<KeyT, 12, 1>(descs, be, b, s, e0, e1); return true;
    case 12 * 4 + 2: launch_rows_tz<KeyT, 12, 2>(descs, be, b, s, e0, e1); return true;
    case 14 * 4 + 1: launch_rows_tz<KeyT, 14, 1>(descs, be, b, s, e0, e1); return true;
    case 14 * 4 + 2: launch_rows_tz<KeyT, 14, 2>(descs, be, b, s, e0, e1); return true;
    case 16 * 4 + 1: launch_rows_tz<KeyT, 16, 1>(descs, be, b, s, e0, e1); return true;
    case 16 * 4 + 2: launch_rows_tz<KeyT, 16, 2>(descs, be, b, s, e0, e1); return true;
    case 24 * 4 + 1: launch_rows_tz<KeyT, 24, 1>(descs, be, b, s, e0, e1); return true;
    case 24 * 4 + 2: launch_rows_tz<KeyT, 24, 2>(descs, be, b, s, e0, e1); return true;
    case 28 * 4 + 1: launch_rows_tz<KeyT, 28, 1>(descs, be, b, s, e0, e1); return true;
    case 28 * 4 + 2: launch_rows_tz<KeyT, 28, 2>(descs, be, b, s, e0, e1); return true;
    default: return false;
    }
}

template <typename KeyT>
static void launch_generic(const GenericArgs *descs, const BatchEntry *be, const Batch &b, hipStream_t s,
                           hipEvent_t e0, hipEvent_t e1) {
    dim3 grid(b.blocks), block(256);
    switch (b.variant) {
    case 1: hipExtLaunchKernelGGL((k_fill_generic<KeyT, 1>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
    case 2: hipExtLaunchKernelGGL((k_fill_generic<KeyT, 2>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
    case 3: hipExtLaunchKernelGGL((k_fill_generic<KeyT, 3>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
    case 4: hipExtLaunchKernelGGL((k_fill_generic<KeyT, 4>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
    case 5: hipExtLaunchKernelGGL((k_fill_generic<KeyT, 5>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
    case 6: hipExtLaunchKernelGGL((k_fill_generic<KeyT, 6>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
    default: hipExtLaunchKernelGGL((k_fill_generic<KeyT, -1>), grid, block, 0, s, e0, e1, 0, descs, be, b.nentries); break;
    }
}


template <typename KeyT>
static pase_status run_search(pase_graph_t g, hipStream_t s, char *ws, uint64_t *min_cost, uint32_t *cfg) {
    DeviceState *d = g->dev;
    Plan &P = g->plan;
    const int n = (int)P.v.size();
    const size_t nv = g->V.size(), ne = g->E.size();

    std::vector<Launch<KeyT>> launches;
    std::vector<Contrib> contrib;
    pase_status st = build_launches<KeyT>(g, ws, launches, contrib);
    if (st != PASE_OK) return st;
    // the dataflow launch needs the resident layout and a kernel variant it
    // carries for every row fill; otherwise the level schedule runs (the
    // resident layout serves it as well)
    bool use_flow = P.resident && g->schedule == kSchedFlow;
    const bool use_lanes = P.resident && (g->schedule == kSchedLanes || g->schedule == kSchedBulk);
    for (int i = 0; i < n && use_flow; i++)
        if (launches[i].rows)
            use_flow = flow_rows_ok(!std::is_same<KeyT, double>::value, P.v[i].TZ, P.v[i].TM,
                                    std::min<uint32_t>(launches[i].ra.na, std::is_same<KeyT, double>::value ? 4 : 7));

    // ---- constant region image (one host-to-device copy)
    char *img = (char *)d->pinned;
    // the layer costs, their device bytes and the split signatures
    // [off_L, off_ovedge) are written by k_cost_tables on the device: unless
    // the caller overrode the costs, that range is not cleared here, and it is
    // left out of the upload once it is large enough to pay for a second copy
    // call (what the one copy then carries there is overwritten on the device)
    const bool upload_costs = g->overridden || P.off_ovedge - P.off_L < (256u << 10);
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
        if (!g->ex_rows[d].empty()) std::memcpy(img + P.off_ex + off, g->ex_rows[d].data(), g->ex_rows[d].size());
        off += g->ex_rows[d].size();
    }
    std::vector<DevVertex> dvs(nv);
    uint64_t loff = 0;
    for (size_t v = 0; v < nv; v++) {
        DevVertex &x = dvs[v];
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
        loff += g->K[v];
    }
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
        sig_off += (uint64_t)g->K[x.src] + g->K[x.dst];
    }
    if (ne) std::memcpy(img + P.off_edge, des.data(), ne * sizeof(DevEdge));
    if (g->overridden) {
        std::memcpy(img + P.off_L, g->ov_layer.data(), g->ov_layer.size() * 8);
        if (!g->ov_edge.empty()) std::memcpy(img + P.off_ovedge, g->ov_edge.data(), g->ov_edge.size() * 8);
    }
    std::memcpy(img + P.off_contrib, contrib.data(), contrib.size() * sizeof(Contrib));
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
    std::memcpy(img + P.off_bt, bt.data(), n * sizeof(BacktrackDesc));

    // ---- batches: per launch slot, one prep launch, one fill launch per kernel
    // variant and one split-reduction launch
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
    BatchEntry *hbe = (BatchEntry *)(img + P.off_batch);
    std::vector<Batch> batches;
    uint32_t nbe = 0;
    // launch groups in enqueue order: the slots (levels, or positions); with
    // lanes, each level's vertices of lane 0, then lane 1, then lane 2
    std::vector<std::vector<int>> groups;
    std::vector<int> group_lane;
    const int nl = use_lanes ? kLanes : 1;
    if (!use_flow) {
        groups.assign((size_t)P.nslots * nl, {});
        group_lane.assign(groups.size(), 0);
        for (int i = 0; i < n; i++) groups[(size_t)P.v[i].slot * nl + (use_lanes ? P.v[i].lane : 0)].push_back(i);
        for (size_t k = 0; k < groups.size(); k++) group_lane[k] = (int)(k % nl);
    }
    int cur_lane = 0, cur_group = 0;
    auto add_batch = [&](Batch::Kind kind, uint32_t variant, const std::vector<int> &members,
                         uint32_t (*nblk)(const Launch<KeyT> &)) {
        if (members.empty()) return;
        Batch b{kind, cur_lane, cur_group, variant, nbe, 0, 0};
        for (int i : members) {
            hbe[nbe].pos = (uint32_t)i;
            hbe[nbe].first = b.blocks;
            hbe[nbe].prio = use_lanes && P.v[i].lane == 1 ? 1u : 0u;
            hbe[nbe].pad = 0;
            b.blocks += nblk(launches[i]);
            nbe++;
            b.nentries++;
        }
        batches.push_back(b);
    };
    // per-group scratch, reused across groups (cleared, capacity kept)
    std::vector<int> prepped, direct, grp;
    std::vector<std::pair<uint32_t, int>> rows, gens, reds;
    std::map<uint32_t, int> shape_dom;   // TZ * 4 + TM -> largest vertex of the group
    for (size_t sl = 0; sl < groups.size(); sl++) {
        const auto &mem = groups[sl];
        cur_lane = group_lane[sl];
        cur_group = (int)sl;
        prepped.clear();
        direct.clear();
        for (int i : mem) (launches[i].direct ? direct : prepped).push_back(i);
        add_batch(Batch::kDirect, 0, direct, [](const Launch<KeyT> &L) { return L.da.nblk; });
        add_batch(Batch::kPrep, 0, prepped, [](const Launch<KeyT> &L) { return L.prep.nwg; });
        rows.clear();
        gens.clear();
        reds.clear();
        // fp64 keys: the row-term count is a kernel template parameter; a
        // small vertex with fewer row terms than the largest vertex of its tile
        // shape in this group gets zero terms appended (each lane adds the
        // zero key once per c) and joins that vertex's launch
        shape_dom.clear();
        for (int i : prepped)
            if (launches[i].rows && std::is_same<KeyT, double>::value) {
                auto it = shape_dom.find(P.v[i].TZ * 4 + P.v[i].TM);
                if (it == shape_dom.end()) shape_dom[P.v[i].TZ * 4 + P.v[i].TM] = i;
                else if (P.v[i].est_us > P.v[it->second].est_us) it->second = i;
            }
        for (int i : prepped) {
            const Launch<KeyT> &L = launches[i];
            if (L.rows) {
                uint32_t na = std::is_same<KeyT, double>::value ? std::min<uint32_t>(L.ra.na, 4) : 7;
                if (std::is_same<KeyT, double>::value && !use_flow) {
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
        std::stable_sort(rows.begin(), rows.end(),
                         [](const std::pair<uint32_t, int> &a, const std::pair<uint32_t, int> &b) { return a.first < b.first; });
        std::stable_sort(gens.begin(), gens.end(),
                         [](const std::pair<uint32_t, int> &a, const std::pair<uint32_t, int> &b) { return a.first < b.first; });
        for (size_t k = 0; k < rows.size();) {
            grp.clear();
            size_t k2 = k;
            for (; k2 < rows.size() && rows[k2].first == rows[k].first; k2++) grp.push_back(rows[k2].second);
            add_batch(Batch::kRows, rows[k].first, grp, [](const Launch<KeyT> &L) { return L.ra.nblocks_launched; });
            k = k2;
        }
        for (size_t k = 0; k < gens.size();) {
            grp.clear();
            size_t k2 = k;
            for (; k2 < gens.size() && gens[k2].first == gens[k].first; k2++) grp.push_back(gens[k2].second);
            add_batch(Batch::kGeneric, gens[k].first, grp, [](const Launch<KeyT> &L) { return L.ga.nblk; });
            k = k2;
        }
        grp.clear();
        for (auto &x : reds) grp.push_back(x.second);
        add_batch(Batch::kReduce, 0, grp, [](const Launch<KeyT> &L) { return L.red.nblk; });
    }
    if (nbe > 3 * (uint64_t)n) return fail(g, PASE_ERR_INTERNAL, "batch table overflow");
    for (const Batch &b : batches)
        if (b.blocks == 0 || b.blocks > 0x7fffffffu) return fail(g, PASE_ERR_TOO_LARGE, "launch grid size");

    // ---- dataflow tables: control block and done counters (zeroed), then the
    // segments of both queues and their dependencies
    FlowPlan fp;
    FlowArgs fa;
    std::memset(&fa, 0, sizeof fa);
    if (use_flow) {
        st = build_flow<KeyT>(g, launches, fp);
        if (st != PASE_OK) return st;
        const uint64_t ctl_bytes = sizeof(FlowCtl) + (4ull * n + 15) / 16 * 16;
        const uint64_t need = ctl_bytes + (fp.seg[0].size() + fp.seg[1].size()) * sizeof(Seg) +
                              fp.deps.size() * sizeof(SegDep);
        if (need > P.flow_bytes) return fail(g, PASE_ERR_INTERNAL, "dataflow table overflow");
        char *fimg = img + P.off_flow;
        std::memset(fimg, 0, ctl_bytes);
        uint64_t o = ctl_bytes;
        for (int q = 0; q < 2; q++) {
            if (!fp.seg[q].empty()) std::memcpy(fimg + o, fp.seg[q].data(), fp.seg[q].size() * sizeof(Seg));
            fa.seg[q] = (const Seg *)(ws + P.off_flow + o);
            fa.nseg[q] = (uint32_t)fp.seg[q].size();
            fa.nitems[q] = fp.nitems[q];
            o += fp.seg[q].size() * sizeof(Seg);
        }
        if (!fp.deps.empty()) std::memcpy(fimg + o, fp.deps.data(), fp.deps.size() * sizeof(SegDep));
        fa.deps = (const SegDep *)(ws + P.off_flow + o);
        fa.ctl = (FlowCtl *)(ws + P.off_flow);
        fa.done = (uint32_t *)(ws + P.off_flow + sizeof(FlowCtl));
    }

    if (upload_costs) {
        HIPCHK(hipMemcpyAsync(ws, img, P.off_cfg, hipMemcpyHostToDevice, s));
    } else {
        HIPCHK(hipMemcpyAsync(ws, img, P.off_L, hipMemcpyHostToDevice, s));
        HIPCHK(hipMemcpyAsync(ws + P.off_ovedge, img + P.off_ovedge, P.off_cfg - P.off_ovedge,
                              hipMemcpyHostToDevice, s));
    }

    const DevVertex *dV = (const DevVertex *)(ws + P.off_vert);
    const DevEdge *dE = (const DevEdge *)(ws + P.off_edge);
    const uint8_t *dex = (const uint8_t *)(ws + P.off_ex);
    uint64_t *dL = (uint64_t *)(ws + P.off_L);
    uint8_t *dls = (uint8_t *)(ws + P.off_lsum);
    uint64_t *dsig = (uint64_t *)(ws + P.off_sig);
    const Contrib *dC = (const Contrib *)(ws + P.off_contrib);
    const PrepArgs *dp = (const PrepArgs *)(ws + P.off_desc);
    const RowsArgs *dr = (const RowsArgs *)(dp + n);
    const GenericArgs *dg = (const GenericArgs *)(dr + n);
    const ReduceArgs *dd = (const ReduceArgs *)(dg + n);
    const DirectArgs *dx = (const DirectArgs *)(dd + n);
    const BatchEntry *dbe = (const BatchEntry *)(ws + P.off_batch);
    uint32_t *dcfg = (uint32_t *)(ws + P.off_cfg);
    SearchOut *dout = (SearchOut *)(ws + P.off_out);

    // fill launches timed with events: every one (profile 1), or only those of
    // the row kernel with a column chunk per lane (profile 2)
    auto timed = [&](const Batch &b) {
        if (g->profile == 1) return b.kind == Batch::kRows || b.kind == Batch::kGeneric || b.kind == Batch::kDirect;
        return g->profile == 2 && b.kind == Batch::kRows && b.variant / 32 != 1;
    };
    uint32_t nfill = use_flow ? 1 : 0;
    for (const Batch &b : batches) nfill += timed(b);
    // the timing events only time the launches they are attached to (read
    // after the search's final synchronization), so they skip the
    // system-scope cache write-back and invalidation a default event performs
    // around the dispatch -- a few microseconds per timed launch otherwise
    if (g->profile && d->ev.size() < 2 * (size_t)nfill) {
        for (size_t k = d->ev.size(); k < 2 * (size_t)nfill; k++) {
            hipEvent_t e;
            HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
            d->ev.push_back(e);
        }
    }
    uint32_t launches_n = 0;
    if (!g->overridden) {
        hipLaunchKernelGGL(k_cost_tables, dim3(grid_for(loff + P.sig_count)), dim3(256), 0, s, dV, (uint32_t)nv,
                           dE, (uint32_t)ne, dex, dL, dls, dsig, loff, P.sig_count, g->r);
        launches_n++;
        if (g->volume && g->mat_total) {
            hipLaunchKernelGGL(k_edge_volume, dim3(grid_for(g->mat_total, 256, 65535)), dim3(256), 0, s, dV, dE,
                               (uint32_t)ne, dex, (uint64_t *)(ws + P.off_vmat), g->mat_total, g->r);
            launches_n++;
        }
    }
    std::vector<int> fill_of(n, -1);   // fill batch of each vertex (profiling)
    uint32_t fb = 0;
    if (use_flow) {
        // every resident workgroup is a worker; at least one per queue
        int &grid = d->flow_grid[std::is_same<KeyT, double>::value ? 0 : 1];
        if (grid == 0) {
            int dev = 0, cus = 0, per_cu = 0;
            HIPCHK(hipGetDevice(&dev));
            HIPCHK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
            HIPCHK(hipDeviceGetAttribute(&d->wall_khz, hipDeviceAttributeWallClockRate, dev));
            HIPCHK(flow_occupancy<KeyT>(&per_cu));
            grid = std::max(2, cus * std::max(1, per_cu));
        }
        const uint64_t items = (uint64_t)fp.nitems[0] + fp.nitems[1];
        const uint32_t G = (uint32_t)std::max<uint64_t>(2, std::min<uint64_t>((uint64_t)grid, items));
        const uint32_t lw = g->lat_workers ? g->lat_workers : G / 16;
        fa.lat_workers = std::max(1u, std::min(G - 1, lw));
        fa.prep = dp;
        fa.rows = dr;
        fa.gen = dg;
        fa.red = dd;
        fa.V = dV;
        fa.E = dE;
        fa.L = dL;
        fa.lsum = dls;
        fa.sig = dsig;
        fa.cb = dC;
        fa.r = g->r;
        // a dependency wait gives up after 10 s plus 100x the planned search time
        double est = 0;
        for (int i = 0; i < n; i++) est += P.v[i].est_us;
        const double hz = 1e3 * (d->wall_khz > 0 ? d->wall_khz : 100000);
        fa.timeout_ticks = (uint64_t)(hz * (10.0 + 100.0 * est * 1e-6));
        hipEvent_t e0 = g->profile ? d->ev[0] : nullptr, e1 = g->profile ? d->ev[1] : nullptr;
        HIPCHK(flow_launch<KeyT>(fa, G, s, e0, e1));
        g->stats.flow_grid = G;
        g->stats.flow_lat_workers = fa.lat_workers;
        g->stats.flow_items = items;
        for (int i = 0; i < n; i++) fill_of[i] = 0;
        fb = 1;
        launches_n++;
    }
    // lanes: every lane starts after the upload and the cost tables; a group
    // (level, lane) waits, per other lane, for the latest level of that lane
    // whose tables it reads (always a lower level: the event is recorded
    // already); the caller's stream joins every lane at the end
    hipStream_t lane_stream[kLanes] = {s, s, s};
    // event of (lane l, level L): lane_ev[1 + L * kLanes + l]; lane_ev[0]: start
    auto lev = [&](int l, int L) { return d->lane_ev[1 + (size_t)L * kLanes + l]; };
    std::vector<std::vector<int>> waited(kLanes, std::vector<int>(kLanes, -1));
    if (use_lanes) {
        for (int l = 1; l < kLanes; l++) {
            if (!d->side[l - 1]) HIPCHK(hipStreamCreateWithFlags(&d->side[l - 1], hipStreamNonBlocking));
            lane_stream[l] = d->side[l - 1];
        }
        const size_t nev = 1 + (size_t)(P.nslots + 1) * kLanes;
        while (d->lane_ev.size() < nev) {
            hipEvent_t e;
            HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableTiming));
            d->lane_ev.push_back(e);
        }
        HIPCHK(hipEventRecord(d->lane_ev[0], s));
        for (int l = 1; l < kLanes; l++) HIPCHK(hipStreamWaitEvent(lane_stream[l], d->lane_ev[0], 0));
    }
    int prev_group = -1;
    for (const Batch &b : batches) {
        const BatchEntry *e = dbe + b.entry0;
        hipStream_t bs = s;
        if (use_lanes) {
            if (b.group != prev_group) {
                if (prev_group >= 0)
                    HIPCHK(hipEventRecord(lev(group_lane[prev_group], prev_group / nl), lane_stream[group_lane[prev_group]]));
                std::vector<int> need(kLanes, -1);
                for (int i : groups[b.group])
                    for (const auto &t : P.v[i].terms)
                        if (P.v[t.j].lane != b.lane) need[P.v[t.j].lane] = std::max(need[P.v[t.j].lane], P.v[t.j].slot);
                for (int l = 0; l < kLanes; l++)
                    if (need[l] > waited[b.lane][l]) {
                        if (need[l] >= b.group / nl)   // a table is read at a later level only
                            return fail(g, PASE_ERR_INTERNAL, "lane wait on a level not enqueued yet");
                        HIPCHK(hipStreamWaitEvent(lane_stream[b.lane], lev(l, need[l]), 0));
                        waited[b.lane][l] = need[l];
                    }
                prev_group = b.group;
            }
            bs = lane_stream[b.lane];
        }
        switch (b.kind) {
        case Batch::kPrep:
            hipLaunchKernelGGL((k_prep<KeyT>), dim3(b.blocks), dim3(kPrepThreads), 0, bs, dp, e, b.nentries, dV, dE,
                               (const uint64_t *)dL, (const uint8_t *)dls, (const uint64_t *)dsig, dC, g->r);
            break;
        case Batch::kRows:
        case Batch::kGeneric:
        case Batch::kDirect:
        {
            // with profiling, the launch itself records its start and end
            // (events attached to the dispatch, no extra packets in the stream)
            const bool tb = timed(b);
            if (tb)
                for (uint32_t k = 0; k < b.nentries; k++) fill_of[hbe[b.entry0 + k].pos] = (int)fb;
            hipEvent_t e0 = tb ? d->ev[2 * fb] : nullptr, e1 = tb ? d->ev[2 * fb + 1] : nullptr;
            if (b.kind == Batch::kRows) {
                if (!launch_rows<KeyT>(dr, e, b, bs, e0, e1)) return fail(g, PASE_ERR_INTERNAL, "no kernel for TZ");
            } else if (b.kind == Batch::kGeneric) {
                launch_generic<KeyT>(dg, e, b, bs, e0, e1);
            } else {
                hipExtLaunchKernelGGL((k_fill_direct<KeyT>), dim3(b.blocks), dim3(256), 0, bs, e0, e1, 0, dx, e,
                                      b.nentries, dV, dE, (const uint64_t *)dL, (const uint8_t *)dls,
                                      (const uint64_t *)dsig, dC, g->r);
            }
            if (tb) fb++;
        }
            break;
        case Batch::kReduce:
            hipLaunchKernelGGL((k_reduce_splits<KeyT>), dim3(b.blocks), dim3(256), 0, bs, dd, e, b.nentries);
            break;
        }
        launches_n++;
    }
    if (use_lanes) {
        // join: the caller's stream waits for the last work of every other lane
        for (int l = 1; l < kLanes; l++) {
            HIPCHK(hipEventRecord(lev(l, P.nslots), lane_stream[l]));
            HIPCHK(hipStreamWaitEvent(s, lev(l, P.nslots), 0));
        }
    }
    const uint32_t *flow_err = use_flow ? &fa.ctl->error : nullptr;
    if ((uint32_t)n <= kMaxBacktrackThreads)
        hipLaunchKernelGGL((k_backtrack_levels<KeyT>), dim3(1), dim3((n + 63) / 64 * 64), 0, s,
                           (const BacktrackDesc *)(ws + P.off_bt), (uint32_t)n, nlev,
                           (const void *)(ws + P.off_T + P.v[n - 1].T_off), dcfg, dout, flow_err);
    else
        hipLaunchKernelGGL((k_backtrack<KeyT>), dim3(1), dim3(64), 0, s, (const BacktrackDesc *)(ws + P.off_bt),
                           (uint32_t)n, (const void *)(ws + P.off_T + P.v[n - 1].T_off), dcfg, dout, flow_err);
    launches_n++;
    HIPCHK(hipGetLastError());
    // the staging buffer is reused for the results: the stream runs the
    // upload before these copies
    char *host_out = img;
    HIPCHK(hipMemcpyAsync(host_out, dout, sizeof(SearchOut), hipMemcpyDeviceToHost, s));
    HIPCHK(hipMemcpyAsync(host_out + sizeof(SearchOut), dcfg, nv * 4, hipMemcpyDeviceToHost, s));
    HIPCHK(hipStreamSynchronize(s));
    SearchOut so;
    std::memcpy(&so, host_out, sizeof so);
    if (so.status & 1u) return fail(g, PASE_ERR_INTERNAL, "a dependency wait of the dataflow launch timed out");
    if (so.status & 2u) return fail(g, PASE_ERR_INTERNAL, "the dataflow launch met an item it cannot run");
    if (so.status) return fail(g, PASE_ERR_INTERNAL, "back-substitution read an argmin out of range");
    *min_cost = so.min_cost;
    std::memcpy(cfg, host_out + sizeof(SearchOut), nv * 4);

    g->stats.launches = launches_n;
    g->stats.slots = (uint32_t)P.nslots;
    if (!use_flow) g->stats.flow_grid = g->stats.flow_lat_workers = 0, g->stats.flow_items = 0;
    g->stats.schedule = use_flow ? 3u : use_lanes ? (uint32_t)g->schedule : (P.by_level ? 0u : 1u);
    g->stats.fill_ms = g->stats.rows_fill_ms = g->stats.stream_fill_ms = 0;
    g->stats.rows_launches = g->stats.stream_launches = 0;
    if (g->profile && use_flow) {
        float ms = 0.f;
        HIPCHK(hipEventElapsedTime(&ms, d->ev[0], d->ev[1]));
        g->stats.fill_ms = g->stats.rows_fill_ms = ms;
        g->stats.rows_launches = 1;
        for (int i = 0; i < n; i++) P.v[i].fill_ms = 0.0;
    } else if (g->profile) {
        std::vector<float> ms(fb, 0.f);
        uint32_t k = 0;
        for (const Batch &b : batches) {
            if (!timed(b)) continue;
            HIPCHK(hipEventElapsedTime(&ms[k], d->ev[2 * k], d->ev[2 * k + 1]));
            g->stats.fill_ms += ms[k];
            if (b.kind == Batch::kRows) {
                g->stats.rows_fill_ms += ms[k];
                g->stats.rows_launches++;
                if (b.variant / 32 == 1) {   // one column per lane: the column-less form
                    g->stats.stream_fill_ms += ms[k];
                    g->stats.stream_launches++;
                }
            }
            k++;
        }
        for (int i = 0; i < n; i++) P.v[i].fill_ms = fill_of[i] >= 0 ? ms[fill_of[i]] : 0.0;
    }
    return PASE_OK;
}

pase_status device_search(pase_graph_t g, void *stream, uint64_t *min_cost, uint32_t *cfg) {
    auto t0 = std::chrono::steady_clock::now();
    pase_status st;
    uint32_t kt = choose_key_type(g, &st);
    if (st != PASE_OK) return fail(g, st, "worst-case key exceeds 64 bits");
    char *ws = nullptr;
    st = ensure_memory(g, &ws);
    if (st != PASE_OK) return st;
    hipStream_t s = (hipStream_t)stream;
    g->searched = false;
    uint64_t mc = 0;
    std::vector<uint32_t> out(g->V.size());
    st = kt == 0 ? run_search<double>(g, s, ws, &mc, out.data()) : run_search<uint64_t>(g, s, ws, &mc, out.data());
    if (st != PASE_OK) return st;
    *min_cost = mc;
    std::memcpy(cfg, out.data(), out.size() * 4);
    g->key_type = kt;
    g->searched = true;
    g->dev->last_stream = s;
    const Plan &P = g->plan;
    g->stats.cells = P.cells;
    g->stats.table_entries = P.entries;
    g->stats.workspace_bytes = P.total;
    g->stats.max_dep = P.max_dep;
    g->stats.key_type = kt;
    g->stats.rows_vertices = P.rows_vertices;
    g->stats.rows_cells = P.rows_cells;
    g->stats.stream_cells = P.stream_cells;
    g->stats.wall_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    return PASE_OK;
}

static char *workspace(pase_graph_t g) {
    DeviceState *d = g->dev;
    return d->lent ? (char *)d->lent : (char *)d->ws;
}

pase_status device_table_entry(pase_graph_t g, int pos, uint64_t idx, uint64_t *cost, uint32_t *arg) {
    const Plan &P = g->plan;
    char *ws = workspace(g);
    const VPlan &vp = P.v[pos];
    uint64_t raw = 0;
    uint16_t a = 0;
    HIPCHK(hipMemcpy(&raw, ws + P.off_T + vp.T_off + idx * 8, 8, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(&a, ws + P.off_A + vp.A_off + idx * 2, 2, hipMemcpyDeviceToHost));
    // tables are stored in their reader's key space (x 2^out_shift)
    if (g->key_type == 0) {
        double dv;
        std::memcpy(&dv, &raw, 8);
        *cost = ((uint64_t)dv) >> vp.out_shift;
    } else {
        *cost = raw >> vp.out_shift;
    }
    *arg = a;
    return PASE_OK;
}

pase_status device_fingerprint(pase_graph_t g, int pos, uint64_t *fpT, uint64_t *fpA) {
    const Plan &P = g->plan;
    char *ws = workspace(g);
    const VPlan &vp = P.v[pos];
    FingerArgs fa;
    std::memset(&fa, 0, sizeof fa);
    fa.T = ws + P.off_T + vp.T_off;
    fa.A = (const uint16_t *)(ws + P.off_A + vp.A_off);
    fa.N = vp.N;
    fa.m = (uint32_t)vp.layout.size();
    fa.out_shift = vp.out_shift;
    // canonical order: D ascending, first digit slowest
    std::vector<uint64_t> cst(vp.D.size(), 1);
    for (int k = (int)vp.D.size() - 2; k >= 0; k--) cst[k] = cst[k + 1] * g->K[vp.D[k + 1]];
    for (size_t k = 0; k < vp.layout.size(); k++) {
        fa.rad[k] = g->K[vp.layout[k]];
        size_t at = std::lower_bound(vp.D.begin(), vp.D.end(), vp.layout[k]) - vp.D.begin();
        fa.cstride[k] = cst[at];
    }
    unsigned long long *dout = nullptr;
    HIPCHK(hipMalloc(&dout, 16));
    HIPCHK(hipMemset(dout, 0, 16));
    fa.out = dout;
    uint32_t grid = grid_for(vp.N, 256, 1024);
    if (g->key_type == 0) hipLaunchKernelGGL(k_fingerprint<double>, dim3(grid), dim3(256), 0, 0, fa);
    else hipLaunchKernelGGL(k_fingerprint<uint64_t>, dim3(grid), dim3(256), 0, 0, fa);
    unsigned long long h[2];
    hipError_t e = hipMemcpy(h, dout, 16, hipMemcpyDeviceToHost);
    (void)hipFree(dout);
    HIPCHK(e);
    *fpT = h[0];
    *fpA = h[1];
    return PASE_OK;
}

pase_status device_layer_costs(pase_graph_t g, uint32_t v, uint64_t *out) {
    const Plan &P = g->plan;
    char *ws = workspace(g);
    uint64_t loff = 0;
    for (uint32_t u = 0; u < v; u++) loff += g->K[u];
    HIPCHK(hipMemcpy(out, ws + P.off_L + loff * 8, (size_t)g->K[v] * 8, hipMemcpyDeviceToHost));
    return PASE_OK;
}

pase_status device_edge_costs(pase_graph_t g, uint32_t e, uint64_t *out) {
    const Plan &P = g->plan;
    char *ws = workspace(g);
    uint64_t n = (uint64_t)g->K[g->E[e].src] * g->K[g->E[e].dst];
    if (g->overridden) {
        HIPCHK(hipMemcpy(out, ws + P.off_ovedge + g->ov_edge_off[e] * 8, n * 8, hipMemcpyDeviceToHost));
        return PASE_OK;
    }
    if (g->volume) {
        HIPCHK(hipMemcpy(out, ws + P.off_vmat + g->mat_off[e] * 8, n * 8, hipMemcpyDeviceToHost));
        return PASE_OK;
    }
    uint64_t *tmp = nullptr;
    HIPCHK(hipMalloc(&tmp, n * 8));
    hipLaunchKernelGGL(k_edge_costs, dim3(grid_for(n)), dim3(256), 0, 0, (const DevVertex *)(ws + P.off_vert),
                       (const DevEdge *)(ws + P.off_edge), e, (const uint8_t *)(ws + P.off_lsum),
                       (const uint64_t *)(ws + P.off_sig), tmp, g->r);
    hipError_t err = hipMemcpy(out, tmp, n * 8, hipMemcpyDeviceToHost);
    (void)hipFree(tmp);
    HIPCHK(err);
    return PASE_OK;
}

}  // namespace pase

template <typename KeyT>
static pase_status flow_check_t(pase_graph_t g, uint32_t workers, uint32_t lat_workers, uint64_t seed,
                                uint64_t *items) {
    // descriptors hold device addresses only: any base will do, nothing is read through it
    char *fake_ws = (char *)(uintptr_t)(1ull << 40);
    std::vector<Launch<KeyT>> launches;
    std::vector<Contrib> contrib;
    pase_status st = build_launches<KeyT>(g, fake_ws, launches, contrib);
    if (st != PASE_OK) return st;
    FlowPlan fp;
    st = build_flow<KeyT>(g, launches, fp);
    if (st != PASE_OK) return st;
    *items = (uint64_t)fp.nitems[0] + fp.nitems[1];
    return flow_simulate(g, fp, workers, lat_workers, seed);
}

extern "C" pase_status pase_flow_check(pase_graph_t g, uint32_t workers, uint32_t lat_workers, uint64_t seed,
                                       uint64_t *items) {
    if (!g || !items || workers < 2 || lat_workers < 1 || lat_workers >= workers)
        return g ? fail(g, PASE_ERR_INVALID_ARGUMENT, "need items, workers >= 2, 1 <= lat_workers < workers")
                 : PASE_ERR_INVALID_ARGUMENT;
    if (!g->planned) return fail(g, PASE_ERR_BAD_STATE, "call pase_enumerate_configs first");
    if (!g->plan.resident || g->schedule != kSchedFlow)
        return fail(g, PASE_ERR_BAD_STATE, "the plan does not use the dataflow schedule");
    pase_status st;
    const uint32_t kt = choose_key_type(g, &st);
    if (st != PASE_OK) return fail(g, st, "worst-case key exceeds 64 bits");
    return kt == 0 ? flow_check_t<double>(g, workers, lat_workers, seed, items)
                   : flow_check_t<uint64_t>(g, workers, lat_workers, seed, items);
}
