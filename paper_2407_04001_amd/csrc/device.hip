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
#include <type_traits>
#include <cstring>
#include <vector>

#include "internal.h"

using namespace pase;

// ------------------------------------------------------------------ key arithmetic
template <typename KeyT> struct KeyOps;

template <> struct KeyOps<double> {
    using Val = double;   // table value type
    static constexpr double sentinel() { return 1152921504606846976.0; }  // 2^60 > any key
    __device__ static double from_u64(uint64_t x) { return (double)x; }
    __device__ static uint64_t val_to_u64(double x) { return (uint64_t)x; }
    __device__ static double add(double a, double b) { return a + b; }
    __device__ static double min(double a, double b) { return __builtin_fmin(a, b); }
    // key = cost * 2^bits + c  ->  (cost * 2^out_shift, c)
    __device__ static void split(double key, uint32_t bits, uint32_t out_shift, double &val, uint32_t &c) {
        double s = __builtin_ldexp(1.0, (int)bits);
        double v = __builtin_trunc(key * __builtin_ldexp(1.0, -(int)bits));
        val = v * __builtin_ldexp(1.0, (int)out_shift);
        c = (uint32_t)__builtin_fma(-v, s, key);
    }
};

template <> struct KeyOps<uint64_t> {
    using Val = uint64_t;
    static constexpr uint64_t sentinel() { return ~0ull; }
    __device__ static uint64_t from_u64(uint64_t x) { return x; }
    __device__ static uint64_t val_to_u64(uint64_t x) { return x; }
    __device__ static uint64_t add(uint64_t a, uint64_t b) { return a + b; }
    __device__ static uint64_t min(uint64_t a, uint64_t b) { return a < b ? a : b; }
    __device__ static void split(uint64_t key, uint32_t bits, uint32_t out_shift, uint64_t &val, uint32_t &c) {
        val = (key >> bits) << out_shift;
        c = (uint32_t)(key & ((1ull << bits) - 1));
    }
};


// Buffer resource word 3 (data format 32-bit, raw addressing) for gfx9-family
// buffer instructions.
constexpr int kBufferWord3 = 0x00020000;

// ------------------------------------------------------------------ cost model (device)
// Layer cost t_l(v, c) = ceil(F / P) + r * (2^e_red - 1) * ceil(keep / 2^(E - e_red)),
// with P = 2^E the device count of the configuration and e_red the exponent
// sum over contracted dims.  Power-of-two divisions are shifts; the host has
// bounded every operand so nothing overflows.
__device__ __forceinline__ uint64_t layer_cost(const DevVertex &dv, const uint8_t *ex, uint64_t r) {
    uint32_t E = 0, ered = 0;
    for (uint32_t k = 0; k < dv.ndims; k++) {
        E += ex[k];
        if ((dv.reduce_mask >> k) & 1u) ered += ex[k];
    }
    uint64_t compute = (dv.flops + ((1ull << E) - 1)) >> E;
    uint32_t ek = E - ered;
    uint64_t part = (dv.keep_n + ((1ull << ek) - 1)) >> ek;
    return compute + r * (((1ull << ered) - 1) * part);
}

// Split signature of one endpoint configuration of an edge: the split
// exponent of every tensor dim (0 for an unsplit dim), 5 bits each.  Two
// endpoints redistribute nothing exactly when their signatures are equal.
__device__ __forceinline__ uint64_t split_signature(const int8_t *dims, uint32_t rank, const uint8_t *ex) {
    uint64_t sig = 0;
    for (uint32_t k = 0; k < rank; k++) sig |= (uint64_t)(dims[k] >= 0 ? ex[dims[k]] : 0) << (5 * k);
    return sig;
}

// Cost tables of the search: layer cost and device count exponent of every
// (vertex, configuration), and the split signatures of every (edge endpoint,
// configuration); r * t_x(e, cu, cv) is then read off two signatures and two
// exponents (edge_cost_sig).
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
            uint32_t E0 = 0;
            for (uint32_t k = 0; k < dv.ndims; k++) E0 += e[k];
            lsum[t] = (uint8_t)E0;
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
                sig[u] = split_signature(de.sdim, de.rank, ex + vs.ex_off + c * vs.ndims);
            } else {
                const DevVertex vd = V[de.dst];
                c -= vs.K;
                sig[u] = split_signature(de.ddim, de.rank, ex + vd.ex_off + c * vd.ndims);
            }
        }
    }
}

__device__ __forceinline__ uint64_t edge_cost_sig(uint64_t sig_a, uint64_t sig_b, uint32_t la, uint32_t lb,
                                                  uint64_t elems, uint64_t r) {
    if (sig_a == sig_b) return 0;
    uint32_t s = la > lb ? la : lb;
    return r * ((elems + ((1ull << s) - 1)) >> s);
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
                               lsum[v.L_off + cv], de.elems, r);
    }
}

// ------------------------------------------------------------------ prep: key-space blocks
// Batched launches: the workgroups of one launch are the concatenation of the
// workgroups of its vertices; find the vertex of this workgroup (uniform).
__device__ __forceinline__ uint32_t batch_find(const BatchEntry *__restrict__ be, uint32_t nbe, uint32_t wg) {
    uint32_t lo = 0, hi = nbe;
    while (hi - lo > 1) {
        uint32_t mid = (lo + hi) >> 1;
        if (be[mid].first <= wg) lo = mid; else hi = mid;
    }
    return __builtin_amdgcn_readfirstlane(lo);
}

// One workgroup handles kPrepThreads consecutive (c, column) elements of one
// outer index of one block, so the block, its contributions and the outer
// digits are uniform across the workgroup (scalar loads); lanes differ only in
// (c, column).
template <typename KeyT>
__global__ __launch_bounds__(kPrepThreads) void k_prep(const PrepArgs *__restrict__ descs,
                                                     const BatchEntry *__restrict__ be, uint32_t nbe,
                                                     const DevVertex *__restrict__ V,
                                                     const DevEdge *__restrict__ E,
                                                     const uint64_t *__restrict__ L,
                                                     const uint8_t *__restrict__ lsum,
                                                     const uint64_t *__restrict__ sig,
                                                     const Contrib *__restrict__ cb, uint64_t r) {
    using Val = typename KeyOps<KeyT>::Val;
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    const PrepArgs &a = descs[be[kb].pos];
    KeyT *__restrict__ blocks = (KeyT *)a.blocks;
    const uint32_t wg = blockIdx.x - be[kb].first;
    uint32_t b = 0;
    while (b + 1 < a.nblocks && wg >= a.blk[b + 1].wg_begin) b++;
    b = __builtin_amdgcn_readfirstlane(b);
    const Block &bk = a.blk[b];
    const uint32_t rel = wg - bk.wg_begin;
    const uint32_t row = rel / bk.chunks, chunk = rel % bk.chunks;
    const uint32_t per_row = a.K * bk.ld;
    const uint32_t e = chunk * kPrepThreads + threadIdx.x;
    if (e >= per_row) return;
    const uint32_t c = e / bk.ld, q = e % bk.ld;
    KeyT *out = blocks + bk.out_off + (uint64_t)row * per_row + e;
    if (bk.post >= 0 && q >= bk.postrad) { *out = (KeyT)0; return; }
    uint32_t dv[kMaxDep];
    for (int k = 0; k < kMaxDep; k++) dv[k] = 0;
    uint32_t x = row;
    for (int k = (int)bk.npre - 1; k >= 0; k--) {
        dv[bk.pre[k]] = x % bk.prerad[k];
        x /= bk.prerad[k];
    }
    if (bk.post >= 0) dv[bk.post] = q;
    const DevVertex me = V[a.vi];
    // plain costs (layer, transfer) are summed in `sum` and shifted into key
    // space at the end; DP tables are stored in this vertex's key space already
    uint64_t sum = 0, keysum = 0, low = 0;
    for (uint32_t k = bk.c_begin; k < bk.c_end; k++) {
        const Contrib ct = cb[k];
        if (ct.kind == kContribLayer) {
            sum += L[me.L_off + c];
            low = c;
        } else if (ct.kind == kContribEdge) {
            const DevEdge de = E[ct.edge];
            const uint32_t xo = dv[ct.dig];
            const DevVertex ov = V[ct.vi_is_src ? de.dst : de.src];
            const uint64_t sme = sig[de.sig_off + (ct.vi_is_src ? 0 : V[de.src].K) + c];
            const uint64_t sot = sig[de.sig_off + (ct.vi_is_src ? me.K : 0) + xo];
            sum += edge_cost_sig(sme, sot, lsum[me.L_off + c], lsum[ov.L_off + xo], de.elems, r);
        } else {
            uint64_t idx = (uint64_t)c * ct.sc;
            for (int k2 = 0; k2 < kMaxDep; k2++) idx += (uint64_t)dv[k2] * ct.sd[k2];
            if (ct.raw_u64) sum += ((const uint64_t *)ct.ptr)[idx];
            else keysum += KeyOps<KeyT>::val_to_u64(((const Val *)ct.ptr)[idx]);
        }
    }
    *out = KeyOps<KeyT>::from_u64((sum << a.bits) + keysum + low);
}

// Waits for every outstanding scalar-memory and LDS read (s_waitcnt
// lgkmcnt(0), other counters left alone).  Scalar loads return out of order,
// so a wait for one of them is always a wait for all of them: the pipelined
// loops wait for the operands of c *before* they request those of c + 1,
// otherwise the wait the compiler places before the first use of c's
// operands would also wait for the prefetch.
__device__ __forceinline__ void wait_lgkm_all() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// ------------------------------------------------------------------ fill: row kernel
// Output T_i is laid out [z][o][r]: column digit z slowest, then the outer
// digits o (those sharing a lookup with z), then the row digits r.  A tile is
// TM x 64 consecutive rows of one (o, column chunk, c range); lane l holds
// rows l, l + 64, ...  For each c every row forms its operand a = sum of its
// row terms, and the wave reads the TZ column operands B[o][c][z0..z0+TZ)
// through the scalar unit (they are wave-uniform), so each cell is one add
// (SGPR operand) and one min; one scalar round trip per c feeds TM x 64 x TZ
// cells.  The four waves of a workgroup take the same tile and a quarter of
// its c range each, and combine their minima through LDS at the end: a wave
// then does a quarter of a tile's work, so a launch has four times as many,
// shorter, work items and its last partial round of waves costs little.
constexpr int kMergeVals = 16;   // values per lane moved through LDS per merge pass

template <typename KeyT, int TZ, int TM, int NA>
__global__ __launch_bounds__(256) void k_fill_rows(const RowsArgs *__restrict__ descs,
                                                  const BatchEntry *__restrict__ be, uint32_t nbe) {
    using Ops = KeyOps<KeyT>;
    using Val = typename Ops::Val;
    __shared__ KeyT xch[2][kMergeVals][64];
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    const RowsArgs &a = descs[be[kb].pos];
    const uint32_t lane = threadIdx.x & 63;
    // the wave index is uniform across the wave: say so, so that everything
    // derived from it (c range, column addresses) lives in SGPRs
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // blocks are dealt round-robin to the 8 XCDs: give every XCD a contiguous
    // range of tiles so that tiles sharing a column slice share an L2 (every
    // vertex's block count and first block are multiples of 8, so the XCD of
    // a block is its local index mod 8)
    const uint32_t nb = a.nblocks_launched, b = blockIdx.x - be[kb].first;
    const uint64_t wg = (uint64_t)(b % 8) * (nb / 8) + b / 8;
    // a workgroup takes 4 / P tiles, P = a.parts waves per tile, each wave a
    // P-th of the tile's c range
    const uint32_t P = a.parts, tpw = 4 / P;
    if (wg * tpw >= a.total_tiles) return;   // the whole workgroup leaves together
    const uint32_t part = wave % P, tin = wave / P;
    const bool has_tile = wg * tpw + tin < a.total_tiles;
    // (a wave without a tile computes nothing but still takes part in the merge)
    const uint64_t tile = min(wg * tpw + tin, a.total_tiles - 1);
    // tile order (fastest first): row tile, column chunk, outer index, c split --
    // all chunks of one outer index run close together and share its slices
    const uint32_t rowtile = (uint32_t)(tile % a.tiles_per_o);
    uint64_t t2 = tile / a.tiles_per_o;
    const uint32_t chunk = (uint32_t)(t2 % a.nchunks);
    t2 /= a.nchunks;
    const uint32_t o = (uint32_t)(t2 % a.MO);
    const uint32_t split = (uint32_t)(t2 / a.MO);

    constexpr int NT = NA < 0 ? kMaxATerms : NA;
    constexpr int NTA = NT > 0 ? NT : 1;
    const int na = NA < 0 ? (int)a.na : NA;
    uint32_t dO[kMaxDep];
    {
        uint32_t x = o;
        for (int k = kMaxDep - 1; k >= 0; k--)
            if (k < (int)a.nO) { dO[k] = x % a.radO[k]; x /= a.radO[k]; } else dO[k] = 0;
    }
    // row terms are read with buffer loads: per-lane byte offset in a VGPR,
    // the c-dependent part as a scalar offset, no per-c address arithmetic
    __amdgpu_buffer_rsrc_t rsrc[NTA];
    uint32_t tsc[NTA];
#pragma unroll
    for (int t = 0; t < NTA; t++) {
        rsrc[t] = __builtin_amdgcn_make_buffer_rsrc(t < na ? const_cast<void *>(a.a[t].ptr) : nullptr, (short)0,
                                                    t < na ? (int)a.a[t].bytes : 0, kBufferWord3);
        tsc[t] = t < na ? a.a[t].sc * (uint32_t)sizeof(Val) : 0;
    }
    uint32_t r[TM], offb[TM][NTA];
    bool valid[TM];
#pragma unroll
    for (int m = 0; m < TM; m++) {
        r[m] = (rowtile * TM + m) * 64 + lane;
        valid[m] = r[m] < a.MR;
        uint32_t x = valid[m] ? r[m] : a.MR - 1, dR[kMaxDep];
        for (int k = kMaxDep - 1; k >= 0; k--)
            if (k < (int)a.nR) { dR[k] = x % a.radR[k]; x /= a.radR[k]; } else dR[k] = 0;
#pragma unroll
        for (int t = 0; t < NTA; t++) {
            uint32_t off = 0;
            if (t < na)
                for (int k = 0; k < kMaxDep; k++) off += dO[k] * a.a[t].sdO[k] + dR[k] * a.a[t].sdR[k];
            offb[m][t] = off * (uint32_t)sizeof(Val);
        }
    }
    // this wave's part [c0, c1) of the tile's c range (possibly empty)
    const uint32_t cs = split * a.cper, ce_ = has_tile ? min(a.K, cs + a.cper) : cs;
    const uint32_t q = (ce_ - cs + P - 1) / P;
    const uint32_t c0 = min(ce_, cs + part * q), c1 = min(ce_, c0 + q);
    const uint32_t ldz = a.ldz;
    const KeyT *B = (const KeyT *)a.B + (uint64_t)o * a.K * ldz + (uint64_t)chunk * TZ;

    KeyT acc[TM][TZ];
#pragma unroll
    for (int m = 0; m < TM; m++)
#pragma unroll
        for (int t = 0; t < TZ; t++) acc[m][t] = Ops::sentinel();

    // Software pipeline over two register sets of U values of c each: the
    // row terms and column chunks of the next U values are requested while
    // the cells of the current ones are computed from the other set, so load
    // latency overlaps VALU work.  Narrow tiles have little work per c and
    // keep U = 4 values in flight per set.  Loads past c1 repeat column
    // c1 - 1 (in bounds, unused) so that every load is unconditional and the
    // register sets never need copying.
    constexpr int U = TZ <= 2 ? 4 : 1;
    using SKey = const __attribute__((address_space(4))) KeyT;
    uint64_t xe[U][TM][NTA], xo[U][TM][NTA];
    KeyT ce[U][TZ], co[U][TZ];
    auto load = [&](uint64_t (&xs)[U][TM][NTA], KeyT (&bs)[U][TZ], uint32_t cc) {
#pragma unroll
        for (int u = 0; u < U; u++) {
            const uint32_t cu = min(cc + u, c1 - 1);
#pragma unroll
            for (int m = 0; m < TM; m++)
#pragma unroll
                for (int t = 0; t < NTA; t++)
                    if (t < na)
                        xs[u][m][t] = __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(
                                                                       rsrc[t], (int)offb[m][t], (int)(cu * tsc[t]), 0));
            SKey *brow = (SKey *)(uintptr_t)(B + (uint64_t)cu * ldz);
#pragma unroll
            for (int t = 0; t < TZ; t++) bs[u][t] = brow[t];
        }
    };
    auto cells = [&](const uint64_t (&xs)[U][TM][NTA], const KeyT (&bs)[U][TZ], uint32_t n) {
#pragma unroll
        for (int u = 0; u < U; u++) {
            if (u > 0 && (uint32_t)u >= n) break;
            KeyT av[TM];
#pragma unroll
            for (int m = 0; m < TM; m++) {
                av[m] = (KeyT)0;
#pragma unroll
                for (int t = 0; t < NTA; t++)
                    if (t < na) {
                        const KeyT v = __builtin_bit_cast(KeyT, xs[u][m][t]);
                        av[m] = t == 0 ? v : Ops::add(av[m], v);
                    }
            }
#pragma unroll
            for (int t = 0; t < TZ; t++)
#pragma unroll
                for (int m = 0; m < TM; m++) acc[m][t] = Ops::min(acc[m][t], Ops::add(av[m], bs[u][t]));
        }
    };
    if (c0 < c1) {
        load(xe, ce, c0);
        uint32_t c = c0;
        for (; c + U < c1; c += 2 * U) {
            // up to 16 columns both sets fit in SGPRs at once: the barriers
            // keep the scheduler from sinking the loads of the next set below
            // the cells of the current one, and the explicit wait for the
            // current operands comes before those loads are issued
            if constexpr (TZ <= 16) {
                wait_lgkm_all();
                __builtin_amdgcn_sched_barrier(0);
            }
            load(xo, co, c + U);
            if constexpr (TZ <= 16) __builtin_amdgcn_sched_barrier(0);
            cells(xe, ce, U);
            if constexpr (TZ <= 16) {
                wait_lgkm_all();
                __builtin_amdgcn_sched_barrier(0);
            }
            load(xe, ce, c + 2 * U);
            if constexpr (TZ <= 16) __builtin_amdgcn_sched_barrier(0);
            cells(xo, co, min((uint32_t)U, c1 - (c + U)));
        }
        if (c < c1) cells(xe, ce, min((uint32_t)U, c1 - c));
    }

    // combine the parts of a tile through LDS, halving the number of holders
    // per stage (P = 4: parts 2, 3 -> 0, 1, then 1 -> 0; P = 2: 1 -> 0),
    // kMergeVals values per lane and pass; P is uniform across the workgroup,
    // so every wave meets the same barriers
    constexpr int V = TM * TZ;
    for (uint32_t d = P / 2; d >= 1; d /= 2) {
#pragma unroll
        for (int p0 = 0; p0 < V; p0 += kMergeVals) {
            constexpr int W = kMergeVals;
            __syncthreads();
            if (part >= d && part < 2 * d) {
                const uint32_t slot = tin * d + (part - d);
#pragma unroll
                for (int j = 0; j < W; j++)
                    if (p0 + j < V) xch[slot][j][lane] = acc[(p0 + j) / TZ][(p0 + j) % TZ];
            }
            __syncthreads();
            if (part < d) {
                const uint32_t slot = tin * d + part;
#pragma unroll
                for (int j = 0; j < W; j++)
                    if (p0 + j < V) {
                        KeyT &x = acc[(p0 + j) / TZ][(p0 + j) % TZ];
                        x = Ops::min(x, xch[slot][j][lane]);
                    }
            }
        }
    }
    if (part != 0 || !has_tile) return;

    const uint64_t plane = (uint64_t)a.MO * a.MR;
    const uint32_t zbase = chunk * TZ;
#pragma unroll
    for (int m = 0; m < TM; m++) {
        if (!valid[m]) continue;
        const uint64_t base_idx = (uint64_t)o * a.MR + r[m];
#pragma unroll
        for (int t = 0; t < TZ; t++) {
            const uint32_t z = zbase + t;
            if (z < a.Kz) {
                const uint64_t idx = (uint64_t)z * plane + base_idx;
                if (a.nsplit > 1) {
                    ((KeyT *)a.partial)[(uint64_t)split * a.N + idx] = acc[m][t];
                } else {
                    Val v;
                    uint32_t cc;
                    Ops::split(acc[m][t], a.bits, a.out_shift, v, cc);
                    ((Val *)a.T)[idx] = v;
                    a.A[idx] = (uint16_t)cc;
                }
            }
        }
    }
}

template <typename KeyT>
__global__ __launch_bounds__(256) void k_reduce_splits(const ReduceArgs *__restrict__ descs,
                                                      const BatchEntry *__restrict__ be, uint32_t nbe) {
    using Ops = KeyOps<KeyT>;
    using Val = typename Ops::Val;
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    const ReduceArgs &a = descs[be[kb].pos];
    const uint32_t lb = blockIdx.x - be[kb].first;
    for (uint64_t t = lb * (uint64_t)blockDim.x + threadIdx.x; t < a.N; t += (uint64_t)a.nblk * blockDim.x) {
        KeyT best = ((const KeyT *)a.partial)[t];
        for (uint32_t s = 1; s < a.nsplit; s++) best = Ops::min(best, ((const KeyT *)a.partial)[s * a.N + t]);
        Val v;
        uint32_t cc;
        Ops::split(best, a.bits, a.out_shift, v, cc);
        ((Val *)a.T)[t] = v;
        a.A[t] = (uint16_t)cc;
    }
}

// ------------------------------------------------------------------ fill: generic kernel
// Any |D(i)| <= PASE_MAX_DEP and any term shapes.  A group of 2^group_log2
// lanes owns one entry phi: lane l evaluates c = l, l + G, ... (key = sum of
// the terms), the group then takes the minimum key with cross-lane swaps.
// Keys are distinct for distinct c, so the minimum -- and with it the lowest
// optimal c -- does not depend on the evaluation order.
template <typename KeyT>
__device__ __forceinline__ KeyT shfl_xor_key(KeyT v, int mask) {
    uint64_t u = __builtin_bit_cast(uint64_t, v);
    uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)u, mask, 64);
    uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(u >> 32), mask, 64);
    return __builtin_bit_cast(KeyT, ((uint64_t)hi << 32) | lo);
}

template <typename KeyT, int NT>
__global__ __launch_bounds__(256) void k_fill_generic(const GenericArgs *__restrict__ descs,
                                                     const BatchEntry *__restrict__ be, uint32_t nbe) {
    using Ops = KeyOps<KeyT>;
    using Val = typename Ops::Val;
    const uint32_t kb = batch_find(be, nbe, blockIdx.x);
    const GenericArgs &a = descs[be[kb].pos];
    const uint32_t lb = blockIdx.x - be[kb].first;
    const uint32_t G = 1u << a.group_log2;
    const uint64_t nthreads = (uint64_t)a.N << a.group_log2;
    constexpr int MT = NT < 0 ? kMaxGTerms : NT;
    const int nt = NT < 0 ? (int)a.nt : NT;
    for (uint64_t tid = lb * (uint64_t)blockDim.x + threadIdx.x; tid < ((nthreads + 255) / 256) * 256;
         tid += (uint64_t)a.nblk * blockDim.x) {
        const bool live = tid < nthreads;
        const uint64_t phi = live ? tid >> a.group_log2 : a.N - 1;
        const uint32_t lane = (uint32_t)(tid & (G - 1));
        uint32_t d[kMaxDep];
        uint64_t x = phi;
        for (int k = kMaxDep - 1; k >= 0; k--)
            if (k < (int)a.m) { d[k] = (uint32_t)(x % a.rad[k]); x /= a.rad[k]; } else d[k] = 0;
        const KeyT *base[MT];
        uint32_t sc[MT];
#pragma unroll
        for (int t = 0; t < MT; t++) {
            uint64_t o = 0;
            if (t < nt)
                for (int k = 0; k < kMaxDep; k++) o += (uint64_t)d[k] * a.t[t].sd[k];
            base[t] = (const KeyT *)a.t[t < nt ? t : 0].ptr + (t < nt ? o : 0);
            sc[t] = t < nt ? a.t[t].sc : 0;
        }
        KeyT best0 = Ops::sentinel(), best1 = Ops::sentinel();
        uint32_t c = lane;
        // two independent chains keep two loads of every term in flight
        for (; c + G < a.K; c += 2 * G) {
            KeyT k0 = base[0][(uint64_t)c * sc[0]];
            KeyT k1 = base[0][(uint64_t)(c + G) * sc[0]];
#pragma unroll
            for (int t = 1; t < MT; t++)
                if (t < nt) {
                    k0 = Ops::add(k0, base[t][(uint64_t)c * sc[t]]);
                    k1 = Ops::add(k1, base[t][(uint64_t)(c + G) * sc[t]]);
                }
            best0 = Ops::min(best0, k0);
            best1 = Ops::min(best1, k1);
        }
        if (c < a.K) {
            KeyT k0 = base[0][(uint64_t)c * sc[0]];
#pragma unroll
            for (int t = 1; t < MT; t++)
                if (t < nt) k0 = Ops::add(k0, base[t][(uint64_t)c * sc[t]]);
            best0 = Ops::min(best0, k0);
        }
        KeyT best = Ops::min(best0, best1);
        for (uint32_t m = G >> 1; m > 0; m >>= 1) best = Ops::min(best, shfl_xor_key(best, (int)m));
        if (live && lane == 0) {
            Val v;
            uint32_t cc;
            Ops::split(best, a.bits, a.out_shift, v, cc);
            ((Val *)a.T)[phi] = v;
            a.A[phi] = (uint16_t)cc;
        }
    }
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
        cfg[d.vi] = d.A[idx];
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
    const uint32_t t = threadIdx.x;
    const bool mine = t < n;
    BacktrackDesc d;
    if (mine) d = bt[t];
    for (uint32_t lev = 0; lev < nlev; lev++) {
        if (mine && d.level == lev) {
            uint64_t idx = 0;
            for (uint32_t k = 0; k < d.m; k++) idx += (uint64_t)scfg[d.dig[k]] * d.stride[k];
            scfg[d.vi] = d.A[idx];
        }
        __syncthreads();
    }
    if (mine) cfg[t] = scfg[t];
    if (t == 0) {
        out->min_cost = KeyOps<KeyT>::val_to_u64(((const typename KeyOps<KeyT>::Val *)Tlast)[0]);
        out->status = 0;
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
    RowsArgs ra;
    GenericArgs ga;
    ReduceArgs red;
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
            if (g->overridden) {
                c.kind = kContribTable;
                c.raw_u64 = 1;
                c.ptr = ovedge + g->ov_edge_off[e];
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
            bk.chunks = (uint32_t)(((uint64_t)vp.K * ld + kPrepThreads - 1) / kPrepThreads);
            bk.wg_begin = L.prep.nwg;
            L.prep.nwg += bk.rows * bk.chunks;
            L.prep.total += bk.elems;
            return (int)L.prep.nblocks++;
        };
        if (vp.kernel == kRows) {
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

// A batched launch: vertices (sequence positions) sharing one kernel variant
// within one launch slot, with their first workgroups.
struct Batch {
    enum Kind { kPrep, kRows, kGeneric, kReduce } kind;
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

    // ---- constant region image (one host-to-device copy)
    char *img = (char *)d->pinned;
    std::memset(img, 0, P.off_cfg);
    uint64_t off = 0;
    std::vector<DevVertex> dvs(nv);
    uint64_t loff = 0;
    for (size_t v = 0; v < nv; v++) {
        std::memcpy(img + P.off_ex + off, g->ex[v].data(), g->ex[v].size());
        DevVertex &x = dvs[v];
        x.ex_off = off;
        x.L_off = loff;
        x.flops = g->flops[v];
        x.keep_n = g->keep_n[v];
        x.K = g->K[v];
        x.ndims = g->V[v].ndims;
        x.reduce_mask = g->V[v].reduce_mask;
        off += g->ex[v].size();
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
        for (uint32_t k = 0; k < kMaxDims; k++) {
            x.sdim[k] = (int8_t)(k < x.rank ? g->E[e].src_dim[k] : -1);
            x.ddim[k] = (int8_t)(k < x.rank ? g->E[e].dst_dim[k] : -1);
        }
        x.elems = g->E[e].elems;
        x.sig_off = sig_off;
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
    for (int i = 0; i < n; i++) {
        hp[i] = launches[i].prep;
        hr[i] = launches[i].ra;
        hg[i] = launches[i].ga;
        hd[i] = launches[i].red;
    }
    BatchEntry *hbe = (BatchEntry *)(img + P.off_batch);
    std::vector<Batch> batches;
    uint32_t nbe = 0;
    std::vector<std::vector<int>> slot_members(P.nslots);
    for (int i = 0; i < n; i++) slot_members[P.v[i].slot].push_back(i);
    auto add_batch = [&](Batch::Kind kind, uint32_t variant, const std::vector<int> &members,
                         uint32_t (*nblk)(const Launch<KeyT> &)) {
        if (members.empty()) return;
        Batch b{kind, variant, nbe, 0, 0};
        for (int i : members) {
            hbe[nbe].pos = (uint32_t)i;
            hbe[nbe].first = b.blocks;
            b.blocks += nblk(launches[i]);
            nbe++;
            b.nentries++;
        }
        batches.push_back(b);
    };
    for (int sl = 0; sl < P.nslots; sl++) {
        const auto &mem = slot_members[sl];
        add_batch(Batch::kPrep, 0, mem, [](const Launch<KeyT> &L) { return L.prep.nwg; });
        std::vector<std::pair<uint32_t, int>> rows, gens, reds;
        for (int i : mem) {
            const Launch<KeyT> &L = launches[i];
            if (L.rows) {
                uint32_t na = std::is_same<KeyT, double>::value ? std::min<uint32_t>(L.ra.na, 4) : 7;
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
            std::vector<int> grp;
            size_t k2 = k;
            for (; k2 < rows.size() && rows[k2].first == rows[k].first; k2++) grp.push_back(rows[k2].second);
            add_batch(Batch::kRows, rows[k].first, grp, [](const Launch<KeyT> &L) { return L.ra.nblocks_launched; });
            k = k2;
        }
        for (size_t k = 0; k < gens.size();) {
            std::vector<int> grp;
            size_t k2 = k;
            for (; k2 < gens.size() && gens[k2].first == gens[k].first; k2++) grp.push_back(gens[k2].second);
            add_batch(Batch::kGeneric, gens[k].first, grp, [](const Launch<KeyT> &L) { return L.ga.nblk; });
            k = k2;
        }
        std::vector<int> rgrp;
        for (auto &x : reds) rgrp.push_back(x.second);
        add_batch(Batch::kReduce, 0, rgrp, [](const Launch<KeyT> &L) { return L.red.nblk; });
    }
    if (nbe > 3 * (uint64_t)n) return fail(g, PASE_ERR_INTERNAL, "batch table overflow");
    for (const Batch &b : batches)
        if (b.blocks == 0 || b.blocks > 0x7fffffffu) return fail(g, PASE_ERR_TOO_LARGE, "launch grid size");

    HIPCHK(hipMemcpyAsync(ws, img, P.off_cfg, hipMemcpyHostToDevice, s));

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
    const BatchEntry *dbe = (const BatchEntry *)(ws + P.off_batch);
    uint32_t *dcfg = (uint32_t *)(ws + P.off_cfg);
    SearchOut *dout = (SearchOut *)(ws + P.off_out);

    uint32_t nfill = 0;
    for (const Batch &b : batches) nfill += b.kind == Batch::kRows || b.kind == Batch::kGeneric;
    if (g->profile && d->ev.size() < 2 * (size_t)nfill) {
        for (size_t k = d->ev.size(); k < 2 * (size_t)nfill; k++) {
            hipEvent_t e;
            HIPCHK(hipEventCreate(&e));
            d->ev.push_back(e);
        }
    }
    uint32_t launches_n = 0;
    if (!g->overridden) {
        hipLaunchKernelGGL(k_cost_tables, dim3(grid_for(loff + P.sig_count)), dim3(256), 0, s, dV, (uint32_t)nv,
                           dE, (uint32_t)ne, dex, dL, dls, dsig, loff, P.sig_count, g->r);
        launches_n++;
    }
    std::vector<int> fill_of(n, -1);   // fill batch of each vertex (profiling)
    uint32_t fb = 0;
    for (const Batch &b : batches) {
        const BatchEntry *e = dbe + b.entry0;
        switch (b.kind) {
        case Batch::kPrep:
            hipLaunchKernelGGL((k_prep<KeyT>), dim3(b.blocks), dim3(kPrepThreads), 0, s, dp, e, b.nentries, dV, dE,
                               (const uint64_t *)dL, (const uint8_t *)dls, (const uint64_t *)dsig, dC, g->r);
            break;
        case Batch::kRows:
        case Batch::kGeneric:
        {
            // with profiling, the launch itself records its start and end
            // (events attached to the dispatch, no extra packets in the stream)
            hipEvent_t e0 = g->profile ? d->ev[2 * fb] : nullptr, e1 = g->profile ? d->ev[2 * fb + 1] : nullptr;
            if (b.kind == Batch::kRows) {
                if (!launch_rows<KeyT>(dr, e, b, s, e0, e1)) return fail(g, PASE_ERR_INTERNAL, "no kernel for TZ");
            } else {
                launch_generic<KeyT>(dg, e, b, s, e0, e1);
            }
        }
            for (uint32_t k = 0; k < b.nentries; k++) fill_of[hbe[b.entry0 + k].pos] = (int)fb;
            fb++;
            break;
        case Batch::kReduce:
            hipLaunchKernelGGL((k_reduce_splits<KeyT>), dim3(b.blocks), dim3(256), 0, s, dd, e, b.nentries);
            break;
        }
        launches_n++;
    }
    if ((uint32_t)n <= kMaxBacktrackThreads)
        hipLaunchKernelGGL((k_backtrack_levels<KeyT>), dim3(1), dim3((n + 63) / 64 * 64), 0, s,
                           (const BacktrackDesc *)(ws + P.off_bt), (uint32_t)n, nlev,
                           (const void *)(ws + P.off_T + P.v[n - 1].T_off), dcfg, dout);
    else
        hipLaunchKernelGGL((k_backtrack<KeyT>), dim3(1), dim3(64), 0, s, (const BacktrackDesc *)(ws + P.off_bt),
                           (uint32_t)n, (const void *)(ws + P.off_T + P.v[n - 1].T_off), dcfg, dout);
    launches_n++;
    HIPCHK(hipGetLastError());
    char *host_out = img;   // reuse the staging buffer after the upload has been consumed
    HIPCHK(hipStreamSynchronize(s));
    HIPCHK(hipMemcpyAsync(host_out, dout, sizeof(SearchOut), hipMemcpyDeviceToHost, s));
    HIPCHK(hipMemcpyAsync(host_out + sizeof(SearchOut), dcfg, nv * 4, hipMemcpyDeviceToHost, s));
    HIPCHK(hipStreamSynchronize(s));
    SearchOut so;
    std::memcpy(&so, host_out, sizeof so);
    if (so.status) return fail(g, PASE_ERR_INTERNAL, "device consistency check failed");
    *min_cost = so.min_cost;
    std::memcpy(cfg, host_out + sizeof(SearchOut), nv * 4);

    g->stats.launches = launches_n;
    g->stats.slots = (uint32_t)P.nslots;
    g->stats.fill_ms = g->stats.rows_fill_ms = g->stats.stream_fill_ms = 0;
    g->stats.rows_launches = g->stats.stream_launches = 0;
    if (g->profile) {
        std::vector<float> ms(fb, 0.f);
        uint32_t k = 0;
        for (const Batch &b : batches) {
            if (b.kind != Batch::kRows && b.kind != Batch::kGeneric) continue;
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
