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
#include <mutex>
#include <string>
#include <type_traits>
#include <cstring>
#include <numeric>
#include <vector>

#include "internal.h"
#include "kernels.h"
#include "launch.h"

using namespace pase;

constexpr uint32_t kSidePrepBlocks = 256;   // grid of a hoisted prep: one workgroup per CU

// Cost tables of the search: layer cost and device byte (device count or its
// log2) of every (vertex, configuration), and the split signatures of every
// (edge endpoint, configuration); r * t_x(e, cu, cv) is then read off two
// signatures and two device bytes (edge_cost_sig).  The same launch sets the
// nF keys of the fused minima to the sentinel `fill` (with caller-given costs
// it runs for that alone, nL = nS = 0).
__global__ void k_cost_tables(const DevVertex *__restrict__ V, uint32_t nv, const DevEdge *__restrict__ E,
                              uint32_t ne, const uint8_t *__restrict__ ex, uint64_t *__restrict__ L,
                              uint8_t *__restrict__ lsum, uint64_t *__restrict__ sig, uint64_t nL,
                              uint64_t nS, uint64_t r, uint64_t *__restrict__ fkeys, uint64_t nF, uint64_t fill) {
    for (uint64_t t = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; t < nL + nS + nF;
         t += (uint64_t)gridDim.x * blockDim.x) {
        if (t >= nL + nS) {
            fkeys[t - nL - nS] = fill;
        } else if (t < nL) {
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
// matrix, into the matrix region the prep kernel then reads like caller-given
// matrices, for every-integer splits (the device walk of volume_cost).  One
// wave per matrix row (grid-stride over the rows of all edges):
// the edge and the producer configuration are uniform, found once per row by
// a scalar search; the lanes take the consumer configurations and write the
// row contiguously.
constexpr int kVolumeThreads = 64;
__global__ __launch_bounds__(kVolumeThreads) void k_edge_volume(const DevVertex *__restrict__ V,
                                                                const DevEdge *__restrict__ E, uint32_t ne,
                                                                const uint8_t *__restrict__ ex,
                                                                uint64_t *__restrict__ out, uint64_t rows,
                                                                uint64_t r) {
    for (uint64_t row = blockIdx.x; row < rows; row += gridDim.x) {
        uint32_t lo = 0, hi = ne;   // last edge with row0 <= row
        while (hi - lo > 1) {
            const uint32_t mid = (lo + hi) / 2;
            if (E[mid].row0 <= row) lo = mid; else hi = mid;
        }
        lo = __builtin_amdgcn_readfirstlane(lo);
        const DevEdge de = E[lo];
        const DevVertex u = V[de.src], v = V[de.dst];
        const uint64_t cu = row - de.row0;
        const uint8_t *exu = ex + u.ex_off + cu * u.ndims;
        uint64_t *o = out + de.mat_off + cu * v.K;
        for (uint32_t cv = threadIdx.x; cv < v.K; cv += kVolumeThreads)
            o[cv] = volume_cost(u, exu, v, ex + v.ex_off + (uint64_t)cv * v.ndims, de, r);
    }
}

// The same for power-of-two splits, which have a closed form.  Every
// coordinate is then a bit field of the device index: tensor dim t's coordinate on u's side is bits
// [o_u, o_u + l_u) of d (o_u = log2 of the splits of the loop dims after the
// mapped one, l_u = log2 of its split), on v's side [o_v, o_v + l_v).  The
// per-dim overlap is min(2^l_u, 2^l_v) when the parts nest -- the top
// w = min(l_u, l_v) bits of both fields agree -- and 0 otherwise, so
// |need n hold| over the devices both ends use (d < 2^n, n = the smaller
// exponent sum; higher bits are zero) is either the product of those minima
// or 0.  The minimum over d is the product iff, for every tensor dim, the
// nested fields coincide for every d: w = 0, the fields start at the same bit
// (o_u + l_u - w = o_v + l_v - w), or both start at bit n or above.  (A
// minimum over d of a conjunction is the conjunction of the minima.)
//
// The producer side of every tensor dim -- its bit field's width and offset --
// is uniform per row and computed once; each lane reads its consumer row's
// exponents into registers.
__global__ __launch_bounds__(kVolumeThreads) void k_edge_volume_pow2(const DevVertex *__restrict__ V,
                                                                     const DevEdge *__restrict__ E, uint32_t ne,
                                                                     const uint8_t *__restrict__ ex,
                                                                     uint64_t *__restrict__ out, uint64_t rows,
                                                                     uint64_t r) {
    for (uint64_t row = blockIdx.x; row < rows; row += gridDim.x) {
        uint32_t lo = 0, hi = ne;   // last edge with row0 <= row
        while (hi - lo > 1) {
            const uint32_t mid = (lo + hi) / 2;
            if (E[mid].row0 <= row) lo = mid; else hi = mid;
        }
        lo = __builtin_amdgcn_readfirstlane(lo);
        const DevEdge &de = E[lo];
        const uint32_t rank = de.rank, du = V[de.src].ndims, dv = V[de.dst].ndims, Kv = V[de.dst].K;
        const uint64_t cu = row - de.row0;
        const uint8_t *exu = ex + V[de.src].ex_off + cu * du;
        // producer side, uniform: exponent sum, and per tensor dim the width and
        // offset of its bit field
        uint32_t nu = 0, lu[kMaxDims], ou[kMaxDims];
#pragma unroll
        for (int k = 0; k < kMaxDims; k++)
            if (k < (int)du) nu += exu[k];
#pragma unroll
        for (int t = 0; t < kMaxDims; t++) {
            lu[t] = ou[t] = 0;
            const int ka = t < (int)rank ? de.sdim[t] : -1;
            if (ka >= 0) {
                lu[t] = exu[ka];
#pragma unroll
                for (int k = 0; k < kMaxDims; k++)
                    if (k > ka && k < (int)du) ou[t] += exu[k];
            }
        }
        const uint64_t elems = de.elems;
        const uint8_t *exv0 = ex + V[de.dst].ex_off;
        uint64_t *o = out + de.mat_off + cu * Kv;
        for (uint32_t cv = threadIdx.x; cv < Kv; cv += kVolumeThreads) {
            const uint8_t *exv = exv0 + (uint64_t)cv * dv;
            uint32_t e[kMaxDims], suffix[kMaxDims + 1];
#pragma unroll
            for (int k = 0; k < kMaxDims; k++) e[k] = k < (int)dv ? exv[k] : 0;
            suffix[kMaxDims] = 0;   // suffix[k] = sum of the exponents of loop dims k..
#pragma unroll
            for (int k = kMaxDims - 1; k >= 0; k--) suffix[k] = suffix[k + 1] + e[k];
            const uint32_t nv = suffix[0], n = nu < nv ? nu : nv;
            uint32_t lq = 0, lneed = 0, lhold = 0, lc = 0;
            bool nested = true;
#pragma unroll
            for (int t = 0; t < kMaxDims; t++) {
                if (t < (int)rank) {
                    const int kb = de.ddim[t];
                    uint32_t lv = 0, ov = 0;
                    // select by an unrolled scan so that e[] and suffix[] stay in registers
#pragma unroll
                    for (int k = 0; k < kMaxDims; k++)
                        if (k == kb) { lv = e[k]; ov = suffix[k + 1]; }
                    const uint32_t w = lu[t] < lv ? lu[t] : lv, fu = ou[t] + lu[t] - w, fv = ov + lv - w;
                    nested &= w == 0 || fu == fv || (fu >= n && fv >= n);
                    lq += lu[t] + lv;
                    lneed += lu[t];
                    lhold += lv;
                    lc += w;
                }
            }
            const uint32_t need_v = 1u << lneed, hold_u = 1u << lhold, m = nested ? 1u << lc : 0;
            const uint32_t fwd = nv > nu ? need_v : need_v - m, bwd = nu > nv ? hold_u : hold_u - m;
            const uint64_t hi_ = elems >> lq, lo_ = elems & ((1ull << lq) - 1), round = (1ull << lq) - 1;
            o[cv] = r * (hi_ * fwd + ((lo_ * fwd + round) >> lq) + hi_ * bwd + ((lo_ * bwd + round) >> lq));
        }
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
                                                     const Contrib *__restrict__ cb, uint64_t r, uint32_t nvb) {
    // nvb work items (the batch's workgroups), grid-stride: a hoisted prep on
    // the side stream runs on a small grid, so that it leaves most CUs to the
    // launches beside it
    for (uint32_t vb = blockIdx.x; vb < nvb; vb += gridDim.x) {
        const uint32_t kb = batch_find(be, nbe, vb);
        set_priority(be[kb]);
        prep_item<KeyT>(descs[be[kb].pos], vb - be[kb].first, V, E, L, lsum, sig, cb, r);
    }
}

template <typename KeyT, int TZ, int TM, int NA>
__global__ __launch_bounds__(256) void k_fill_rows(const RowsArgs *__restrict__ descs,
                                                  const GenericArgs *__restrict__ gdescs,
                                                  const BatchEntry *__restrict__ be, uint32_t nbe) {
    __shared__ MergeBuf<KeyT> xch;
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    set_priority(be[kb]);
    // a small two-term generic fill of the same level rides along in this
    // launch instead of a launch of its own (its workgroups use no LDS and no
    // barrier, and need fewer registers than the row fill)
    if (be[kb].kind == kEntryGeneric2) {
        generic_item<KeyT, 2>(gdescs[be[kb].pos], blockIdx.x - be[kb].first);
        return;
    }
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
    __shared__ KeyT xch[4];   // per-wave minima of a group of several waves
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    set_priority(be[kb]);
    direct_item<KeyT>(descs[be[kb].pos], blockIdx.x - be[kb].first, V, E, L, lsum, sig, cb, r, xch);
}

// ------------------------------------------------------------------ back-substitution
// From the last position down: the configuration of v_i is A_i at the
// already-chosen configurations of D(i) (every member of D(i) is later in the
// sequence).  Single thread; n dependent reads.
template <typename KeyT>
__global__ void k_backtrack(const BacktrackDesc *__restrict__ bt, uint32_t n, const void *Tlast,
                            uint32_t *__restrict__ cfg, SearchOut *out) {
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
    out->status = status;
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
                                                                          SearchOut *out) {
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
        out->status = sbad;
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
        st += splitmix64_mix(h ^ KeyOps<KeyT>::unshift(((const Val *)a.T)[t], a.out_shift));
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

struct DeviceState {
    void *ws = nullptr;
    uint64_t ws_bytes = 0;
    bool owned = false;
    void *pinned = nullptr;
    uint64_t pinned_bytes = 0;
    std::vector<hipEvent_t> ev;        // profiling: two per timed fill launch
    hipEvent_t phase_ev[4] = {};       // profiling: search phases (cost tables | fill | back-substitution)
    hipStream_t last_stream = nullptr;
    char *last_ws = nullptr;           // workspace of the last search (its tables are read there)
    hipStream_t side = nullptr;        // lanes: lane 1's stream; level layout: hoisted preps
                                       // (default priority, as every stream here)
    std::vector<hipEvent_t> lane_ev;   // bulk lane schedule: joins (no timing)
    std::vector<hipEvent_t> hoist_ev;  // hoisted preps: per side batch, its start and its end (no timing)
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
    for (auto e : d->hoist_ev) (void)hipEventDestroy(e);
    for (auto e : d->phase_ev)
        if (e) (void)hipEventDestroy(e);
    if (d->side) (void)hipStreamDestroy(d->side);
    delete d;
    g->dev = nullptr;
}

static DeviceState *state(pase_graph_t g) {
    if (!g->dev) g->dev = new DeviceState();
    return g->dev;
}

static pase_status ensure_memory(pase_graph_t g, char **ws) {
    DeviceState *d = state(g);
    const uint64_t need = g->plan.total;
    if (g->lent_ws) {
        *ws = (char *)g->lent_ws;   // its size was checked before any device work
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

template <typename KeyT, int TZ, int TM>
static void launch_rows_tz(const RowsArgs *descs, const GenericArgs *gdescs, const BatchEntry *be, const Batch &b,
                           hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    dim3 grid(b.blocks), block(256);
    const uint32_t na = b.variant % 8;
    if constexpr (std::is_same<KeyT, double>::value) {
        switch (na) {
        case 0: hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, 0>), grid, block, 0, s, e0, e1, 0, descs, gdescs, be, b.nentries); break;
        case 1: hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, 1>), grid, block, 0, s, e0, e1, 0, descs, gdescs, be, b.nentries); break;
        case 2: hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, 2>), grid, block, 0, s, e0, e1, 0, descs, gdescs, be, b.nentries); break;
        case 3: hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, 3>), grid, block, 0, s, e0, e1, 0, descs, gdescs, be, b.nentries); break;
        default: hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, 4>), grid, block, 0, s, e0, e1, 0, descs, gdescs, be, b.nentries); break;
        }
    } else {
        hipExtLaunchKernelGGL((k_fill_rows<KeyT, TZ, TM, -1>), grid, block, 0, s, e0, e1, 0, descs, gdescs, be,
                              b.nentries);
    }
}

// variant = (TZ * 4 + TM) * 8 + NA
template <typename KeyT>
static bool launch_rows(const RowsArgs *descs, const GenericArgs *gdescs, const BatchEntry *be, const Batch &b,
                        hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    switch (b.variant / 8) {
    case 1 * 4 + 1: launch_rows_tz<KeyT, 1, 1>(descs, gdescs, be, b, s, e0, e1); return true;
    case 1 * 4 + 2: launch_rows_tz<KeyT, 1, 2>(descs, gdescs, be, b, s, e0, e1); return true;
    case 8 * 4 + 1: launch_rows_tz<KeyT, 8, 1>(descs, gdescs, be, b, s, e0, e1); return true;
    case 8 * 4 + 2: launch_rows_tz<KeyT, 8, 2>(descs, gdescs, be, b, s, e0, e1); return true;
    case 12 * 4 + 1: launch_rows_tz<KeyT, 12, 1>(descs, gdescs, be, b, s, e0, e1); return true;
    case 12 * 4 + 2: launch_rows_tz<KeyT, 12, 2>(descs, gdescs, be, b, s, e0, e1); return true;
    case 14 * 4 + 1: launch_rows_tz<KeyT, 14, 1>(descs, gdescs, be, b, s, e0, e1); return true;
    case 14 * 4 + 2: launch_rows_tz<KeyT, 14, 2>(descs, gdescs, be, b, s, e0, e1); return true;
    case 16 * 4 + 1: launch_rows_tz<KeyT, 16, 1>(descs, gdescs, be, b, s, e0, e1); return true;
    case 16 * 4 + 2: launch_rows_tz<KeyT, 16, 2>(descs, gdescs, be, b, s, e0, e1); return true;
    case 24 * 4 + 1: launch_rows_tz<KeyT, 24, 1>(descs, gdescs, be, b, s, e0, e1); return true;
    case 24 * 4 + 2: launch_rows_tz<KeyT, 24, 2>(descs, gdescs, be, b, s, e0, e1); return true;
    case 28 * 4 + 1: launch_rows_tz<KeyT, 28, 1>(descs, gdescs, be, b, s, e0, e1); return true;
    case 28 * 4 + 2: launch_rows_tz<KeyT, 28, 2>(descs, gdescs, be, b, s, e0, e1); return true;
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


// One search on stream s with the workspace at device address ws and the
// host staging buffer img (at least plan.off_cfg bytes).  noalloc: create no
// stream or event (profiling off, one stream).
template <typename KeyT>
static pase_status run_search(pase_graph_t g, hipStream_t s, char *ws, char *img, bool noalloc, uint64_t *min_cost,
                              uint32_t *cfg) {
    DeviceState *d = g->dev;
    Plan &P = g->plan;
    const int n = (int)P.v.size();
    const size_t nv = g->V.size(), ne = g->E.size();
    const auto t_setup = std::chrono::steady_clock::now();
    constexpr bool kWide = std::is_same<KeyT, u128>::value;   // 128-bit keys: prep + generic fills only

    // ---- constant region image and batched launches (host), one upload
    SearchImage si;
    pase_status st = build_image<KeyT>(g, ws, img, si, !noalloc);
    if (st != PASE_OK) return st;
    g->stats.setup_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_setup).count();
    const std::vector<Batch> &batches = si.batches;
    if (si.upload_costs) {
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
    const int profile = noalloc ? 0 : g->profile;
    auto timed = [&](const Batch &b) {
        if (profile == 1) return b.kind == Batch::kRows || b.kind == Batch::kGeneric || b.kind == Batch::kDirect;
        return profile == 2 && b.kind == Batch::kRows && b.variant / 32 != 1;
    };
    uint32_t nfill = 0;
    for (const Batch &b : batches) nfill += timed(b);
    // the timing events only time the launches they are attached to (read
    // after the search's final synchronization), so they skip the
    // system-scope cache write-back and invalidation a default event performs
    // around the dispatch -- a few microseconds per timed launch otherwise
    if (profile) {
        for (size_t k = d->ev.size(); k < 2 * (size_t)nfill; k++) {
            hipEvent_t e;
            HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
            d->ev.push_back(e);
        }
        for (auto &e : d->phase_ev)
            if (!e) HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
        HIPCHK(hipEventRecord(d->phase_ev[0], s));
    }
    uint32_t launches_n = 0;
    // keys of the fused minima start at the sentinel (the bit pattern of the
    // key type's sentinel: keys are non-negative, so 64-bit patterns order like them)
    uint64_t nF = 0, fsent = 0;
    if constexpr (!kWide) {
        nF = P.fused_bytes / 8;
        const KeyT sk = KeyOps<KeyT>::sentinel();
        std::memcpy(&fsent, &sk, 8);
    }
    uint64_t *dfk = (uint64_t *)(ws + P.off_fused);
    if (g->overridden && nF) {
        hipLaunchKernelGGL(k_cost_tables, dim3(grid_for(nF)), dim3(256), 0, s, dV, (uint32_t)nv, dE, (uint32_t)ne, dex,
                           dL, dls, dsig, (uint64_t)0, (uint64_t)0, g->r, dfk, nF, fsent);
        launches_n++;
    }
    if (!g->overridden) {
        hipLaunchKernelGGL(k_cost_tables, dim3(grid_for(si.nL + P.sig_count + nF)), dim3(256), 0, s, dV,
                           (uint32_t)nv, dE, (uint32_t)ne, dex, dL, dls, dsig, si.nL, P.sig_count, g->r, dfk, nF,
                           fsent);
        launches_n++;
        if (g->volume && g->mat_total) {
            hipLaunchKernelGGL(g->factors ? k_edge_volume : k_edge_volume_pow2, dim3(grid_for(g->mat_rows, 1, 65535)),
                               dim3(kVolumeThreads), 0, s, dV, dE, (uint32_t)ne, dex, (uint64_t *)(ws + P.off_vmat),
                               g->mat_rows, g->r);
            launches_n++;
        }
    }
    if (profile) HIPCHK(hipEventRecord(d->phase_ev[1], s));
    std::vector<int> fill_of(n, -1);   // timed fill batch of each vertex (profiling)
    uint32_t fb = 0;
    // bulk lane schedule: the bulk stream starts after the upload and the cost
    // tables; a group (slot, lane) waits, for the other lane, for the latest
    // slot of that lane whose tables it reads (always an earlier slot: its
    // event is recorded already); the caller's stream joins the bulk stream at
    // the end
    const int nl = si.lanes ? kLanes : 1;
    hipStream_t lane_stream[kLanes];
    for (auto &ls : lane_stream) ls = s;
    // event of (lane l, slot L): lane_ev[1 + L * kLanes + l]; lane_ev[0]: start
    auto lev = [&](int l, int L) { return d->lane_ev[1 + (size_t)L * kLanes + l]; };
    int waited[kLanes][kLanes];
    for (auto &row : waited)
        for (int &w : row) w = -1;
    std::vector<char> lane_ev_used;
    if (si.lanes) {
        if (!d->side) HIPCHK(hipStreamCreateWithFlags(&d->side, hipStreamNonBlocking));
        lane_stream[1] = d->side;
        const size_t nev = 1 + (size_t)(P.nslots + 1) * kLanes;
        while (d->lane_ev.size() < nev) {
            hipEvent_t e;
            HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableTiming));
            d->lane_ev.push_back(e);
        }
        HIPCHK(hipEventRecord(d->lane_ev[0], s));
        for (int l = 1; l < kLanes; l++)
            if (lane_stream[l] != s) HIPCHK(hipStreamWaitEvent(lane_stream[l], d->lane_ev[0], 0));
        // a group's event is recorded only when a group of the other lane
        // waits on it: a record is a packet of its own in the lane's queue,
        // which the next kernel of that lane waits behind
        lane_ev_used.assign(nev, 0);
        for (size_t gi = 0; gi < si.groups.size(); gi++) {
            const int ln = si.group_lane[gi];
            for (int i : si.groups[gi])
                for (const auto &t : P.v[i].terms)
                    if (P.v[t.j].lane != ln) lane_ev_used[1 + (size_t)P.v[t.j].slot * kLanes + P.v[t.j].lane] = 1;
        }
    }
    // hoisted preps: a side batch starts after everything enqueued on s before
    // it (the fills of the tables it reads) and its vertex's group waits for it
    std::vector<int> side_of(batches.size(), -1);
    if (si.hoist) {
        if (!d->side) HIPCHK(hipStreamCreateWithFlags(&d->side, hipStreamNonBlocking));
        size_t nside = 0;
        for (const Batch &b : batches) nside += b.side;
        while (d->hoist_ev.size() < 2 * nside) {
            hipEvent_t e;
            HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableTiming));
            d->hoist_ev.push_back(e);
        }
    }
    int nside_done = 0, waits_group = -1;
    int prev_group = -1;
    for (size_t bi = 0; bi < batches.size(); bi++) {
        const Batch &b = batches[bi];
        const BatchEntry *e = dbe + b.entry0;
        hipStream_t bs = s;
        if (si.hoist) {
            if (b.side) {
                hipEvent_t e0 = d->hoist_ev[2 * nside_done], e1 = d->hoist_ev[2 * nside_done + 1];
                HIPCHK(hipEventRecord(e0, s));
                HIPCHK(hipStreamWaitEvent(d->side, e0, 0));
                hipLaunchKernelGGL((k_prep<KeyT>), dim3(std::min<uint32_t>(b.blocks, kSidePrepBlocks)), dim3(kPrepThreads),
                                   0, d->side, dp, e, b.nentries, dV, dE, (const uint64_t *)dL, (const uint8_t *)dls,
                                   (const uint64_t *)dsig, dC, g->r, b.blocks);
                HIPCHK(hipEventRecord(e1, d->side));
                side_of[bi] = nside_done++;
                launches_n++;
                continue;
            }
            if (b.group != waits_group) {
                for (int sb : si.group_waits[(size_t)b.group]) {
                    if (sb < 0 || (size_t)sb >= bi || side_of[sb] < 0)
                        return fail(g, PASE_ERR_INTERNAL, "wait on a hoisted prep not enqueued yet");
                    HIPCHK(hipStreamWaitEvent(s, d->hoist_ev[2 * side_of[sb] + 1], 0));
                }
                waits_group = b.group;
            }
        }
        if (si.lanes) {
            if (b.group != prev_group) {
                if (prev_group >= 0 &&
                    lane_ev_used[1 + (size_t)(prev_group / nl) * kLanes + si.group_lane[prev_group]])
                    HIPCHK(hipEventRecord(lev(si.group_lane[prev_group], prev_group / nl),
                                          lane_stream[si.group_lane[prev_group]]));
                int need[kLanes];
                for (int &x : need) x = -1;
                for (int i : si.groups[b.group])
                    for (const auto &t : P.v[i].terms)
                        if (P.v[t.j].lane != b.lane) need[P.v[t.j].lane] = std::max(need[P.v[t.j].lane], P.v[t.j].slot);
                for (int l = 0; l < kLanes; l++)
                    if (need[l] > waited[b.lane][l]) {
                        if (need[l] >= b.group / nl)   // a table is read at a later slot only
                            return fail(g, PASE_ERR_INTERNAL, "lane wait on a slot not enqueued yet");
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
                               (const uint64_t *)dL, (const uint8_t *)dls, (const uint64_t *)dsig, dC, g->r, b.blocks);
            break;
        case Batch::kRows:
        case Batch::kGeneric:
        case Batch::kDirect:
        {
            // with profiling, the launch itself records its start and end
            // (events attached to the dispatch, no extra packets in the stream)
            const bool tb = timed(b);
            if (tb)
                for (uint32_t k = 0; k < b.nentries; k++) fill_of[((const BatchEntry *)(img + P.off_batch))[b.entry0 + k].pos] = (int)fb;
            hipEvent_t e0 = tb ? d->ev[2 * fb] : nullptr, e1 = tb ? d->ev[2 * fb + 1] : nullptr;
            if (b.kind == Batch::kGeneric) {
                launch_generic<KeyT>(dg, e, b, bs, e0, e1);
            } else if constexpr (kWide) {
                return fail(g, PASE_ERR_INTERNAL, "a 128-bit key plan holds a row or direct fill");
            } else if (b.kind == Batch::kRows) {
                if (!launch_rows<KeyT>(dr, dg, e, b, bs, e0, e1)) return fail(g, PASE_ERR_INTERNAL, "no kernel for TZ");
            } else {
                hipExtLaunchKernelGGL((k_fill_direct<KeyT>), dim3(b.blocks), dim3(256), 0, bs, e0, e1, 0, dx, e,
                                      b.nentries, dV, dE, (const uint64_t *)dL, (const uint8_t *)dls,
                                      (const uint64_t *)dsig, dC, g->r);
            }
            if (tb) fb++;
        }
            break;
        case Batch::kReduce:
            if constexpr (kWide) {
                return fail(g, PASE_ERR_INTERNAL, "a 128-bit key plan holds a split reduction");
            } else {
                hipLaunchKernelGGL((k_reduce_splits<KeyT>), dim3(b.blocks), dim3(256), 0, bs, dd, e, b.nentries);
            }
            break;
        }
        launches_n++;
    }
    if (si.lanes) {
        // join: the caller's stream waits for the last work of the other lanes
        for (int l = 1; l < kLanes; l++)
            if (lane_stream[l] != s) {
                HIPCHK(hipEventRecord(lev(l, P.nslots), lane_stream[l]));
                HIPCHK(hipStreamWaitEvent(s, lev(l, P.nslots), 0));
            }
    }
    if (profile) HIPCHK(hipEventRecord(d->phase_ev[2], s));
    if ((uint32_t)n <= kMaxBacktrackThreads)
        hipLaunchKernelGGL((k_backtrack_levels<KeyT>), dim3(1), dim3((n + 63) / 64 * 64), 0, s,
                           (const BacktrackDesc *)(ws + P.off_bt), (uint32_t)n, si.nlev,
                           (const void *)(ws + P.off_T + P.v[n - 1].T_off), dcfg, dout);
    else
        hipLaunchKernelGGL((k_backtrack<KeyT>), dim3(1), dim3(64), 0, s, (const BacktrackDesc *)(ws + P.off_bt),
                           (uint32_t)n, (const void *)(ws + P.off_T + P.v[n - 1].T_off), dcfg, dout);
    launches_n++;
    if (profile) HIPCHK(hipEventRecord(d->phase_ev[3], s));
    HIPCHK(hipGetLastError());
    // the staging buffer is reused for the results: the stream runs the
    // upload before this copy.  The strategy and the search output are
    // adjacent in the workspace ([off_cfg, off_out + sizeof(SearchOut))), so
    // one copy brings both back
    char *host_out = img;
    const uint64_t out_bytes = P.off_out - P.off_cfg + sizeof(SearchOut);
    // (the staging buffer holds at least max(off_cfg, 4096) bytes)
    if (out_bytes > std::max<uint64_t>(P.off_cfg, 4096)) return fail(g, PASE_ERR_INTERNAL, "result staging size");
    HIPCHK(hipMemcpyAsync(host_out, dcfg, out_bytes, hipMemcpyDeviceToHost, s));
    HIPCHK(hipStreamSynchronize(s));
    SearchOut so;
    std::memcpy(&so, host_out + (P.off_out - P.off_cfg), sizeof so);
    if (so.status) return fail(g, PASE_ERR_INTERNAL, "back-substitution read an argmin out of range");
    *min_cost = so.min_cost;
    std::memcpy(cfg, host_out, nv * 4);

    g->stats.launches = launches_n;
    g->stats.slots = (uint32_t)P.nslots;
    g->stats.schedule = si.lanes ? (uint32_t)g->schedule : (P.by_level ? (uint32_t)kSchedLevel : (uint32_t)kSchedSeq);
    g->stats.fill_ms = g->stats.rows_fill_ms = g->stats.stream_fill_ms = 0;
    g->stats.cost_tables_ms = g->stats.fill_span_ms = g->stats.backtrack_ms = 0;
    g->stats.rows_launches = g->stats.stream_launches = 0;
    if (profile) {
        float ph[3] = {0.f, 0.f, 0.f};
        for (int k = 0; k < 3; k++) HIPCHK(hipEventElapsedTime(&ph[k], d->phase_ev[k], d->phase_ev[k + 1]));
        g->stats.cost_tables_ms = ph[0];
        g->stats.fill_span_ms = ph[1];
        g->stats.backtrack_ms = ph[2];
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

// The search itself, once the workspace (device) and staging buffer (host)
// are known; records the statistics and the workspace the tables live in.
static pase_status search_in(pase_graph_t g, hipStream_t s, char *ws, char *img, bool noalloc, uint32_t kt,
                             std::chrono::steady_clock::time_point t0, uint64_t *min_cost, uint32_t *cfg) {
    g->searched = false;
    uint64_t mc = 0;
    std::vector<uint32_t> out(g->V.size());
    pase_status st = kt == 0   ? run_search<double>(g, s, ws, img, noalloc, &mc, out.data())
                     : kt == 1 ? run_search<uint64_t>(g, s, ws, img, noalloc, &mc, out.data())
                               : run_search<u128>(g, s, ws, img, noalloc, &mc, out.data());
    if (st != PASE_OK) return st;
    *min_cost = mc;
    std::memcpy(cfg, out.data(), out.size() * 4);
    g->key_type = kt;
    g->searched = true;
    g->dev->last_stream = s;
    g->dev->last_ws = ws;
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

// The key type of the plan (R10), decided when the plan was made.
static pase_status plan_keys(pase_graph_t g, uint32_t *kt) {
    pase_status st;
    *kt = choose_key_type(g, &st);
    if (st != PASE_OK) return fail(g, st, "a cost bound of the recurrence exceeds 64 bits");
    if (*kt != g->plan_key_type || (*kt == 2) != g->plan_wide)
        return fail(g, PASE_ERR_INTERNAL, "key type differs from the plan's");
    return PASE_OK;
}

pase_status device_search(pase_graph_t g, void *stream, uint64_t *min_cost, uint32_t *cfg) {
    const auto t0 = std::chrono::steady_clock::now();
    uint32_t kt = 0;
    pase_status st = plan_keys(g, &kt);
    if (st != PASE_OK) return st;
    char *ws = nullptr;
    st = ensure_memory(g, &ws);
    if (st != PASE_OK) return st;
    return search_in(g, (hipStream_t)stream, ws, (char *)g->dev->pinned, false, kt, t0, min_cost, cfg);
}

// ------------------------------------------------------------------ allocation-free search
// The workspace of pase_find_best_strategy_noalloc: one static array that
// every GPU the library runs on holds for the life of the process, each at
// its own address.  In host code `scratch` only names the symbol: its device
// address on the current GPU comes from hipGetSymbolAddress, once per device,
// and only that address is ever handed to a kernel or a copy.
constexpr uint64_t kScratchBytes = PASE_NOALLOC_WORKSPACE_BYTES;
constexpr int kScratchDevices = 64;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {
std::mutex g_scratch_mu;                        // one allocation-free search at a time per process
char *g_scratch_ptr[kScratchDevices] = {};      // device address of `scratch` per device
alignas(256) char g_scratch_img[kScratchBytes]; // host staging of the constant region
}  // namespace

pase_status device_search_noalloc(pase_graph_t g, void *stream, uint64_t *min_cost, uint32_t *cfg) {
    const auto t0 = std::chrono::steady_clock::now();
    uint32_t kt = 0;
    const pase_status st = plan_keys(g, &kt);
    if (st != PASE_OK) return st;
    if (g->plan.total > kScratchBytes)
        return fail(g, PASE_ERR_TOO_LARGE,
                    "the search needs " + std::to_string(g->plan.total) + " bytes of device memory, more than the " +
                        std::to_string(kScratchBytes) + " of the allocation-free workspace");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    int dev = 0;
    HIPCHK(hipGetDevice(&dev));
    if (dev < 0 || dev >= kScratchDevices) return fail(g, PASE_ERR_INVALID_ARGUMENT, "device index out of range");
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        HIPCHK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p || (uintptr_t)p % 256) return fail(g, PASE_ERR_INTERNAL, "static workspace address");
        g_scratch_ptr[dev] = (char *)p;
    }
    state(g);
    return search_in(g, (hipStream_t)stream, g_scratch_ptr[dev], g_scratch_img, true, kt, t0, min_cost, cfg);
}

// The workspace the last search ran in (library-owned, lent or static).
static char *workspace(pase_graph_t g) { return g->dev->last_ws; }

pase_status device_table_entry(pase_graph_t g, int pos, uint64_t idx, uint64_t *cost, uint32_t *arg) {
    const Plan &P = g->plan;
    char *ws = workspace(g);
    const VPlan &vp = P.v[pos];
    const uint64_t kb = key_bytes(g);
    unsigned char raw[16] = {0};
    uint16_t a = 0;
    HIPCHK(hipMemcpy(raw, ws + P.off_T + vp.T_off + idx * kb, kb, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(&a, ws + P.off_A + vp.A_off + idx * 2, 2, hipMemcpyDeviceToHost));
    // tables are stored in their reader's key space (x 2^out_shift)
    if (g->key_type == 0) {
        double dv;
        std::memcpy(&dv, raw, 8);
        *cost = ((uint64_t)dv) >> vp.out_shift;
    } else if (g->key_type == 1) {
        uint64_t x;
        std::memcpy(&x, raw, 8);
        *cost = x >> vp.out_shift;
    } else {
        unsigned __int128 x;
        std::memcpy(&x, raw, 16);
        *cost = (uint64_t)(x >> vp.out_shift);
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
    else if (g->key_type == 1) hipLaunchKernelGGL(k_fingerprint<uint64_t>, dim3(grid), dim3(256), 0, 0, fa);
    else hipLaunchKernelGGL(k_fingerprint<u128>, dim3(grid), dim3(256), 0, 0, fa);
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
