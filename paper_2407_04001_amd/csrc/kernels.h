// Device code of the kernels of libpase (gfx950): key arithmetic, the device
// cost model, and the work of one workgroup of each kernel ("items").
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "internal.h"

namespace pase {

// ------------------------------------------------------------------ key arithmetic
template <typename KeyT> struct KeyOps;

// Val: the type of a stored table value (cost x 2^out_shift, in its reader's
// key space); Acc: an exact integer wide enough for one key, in which prep
// sums its contributions before the key is formed.
template <> struct KeyOps<double> {
    using Val = double;   // table value type
    using Acc = uint64_t;
    static constexpr double sentinel() { return 1152921504606846976.0; }  // 2^60 > any key
    __device__ static double from_u64(uint64_t x) { return (double)x; }
    __device__ static double from_acc(uint64_t x) { return (double)x; }
    __device__ static uint64_t val_to_u64(double x) { return (uint64_t)x; }
    __device__ static uint64_t val_to_acc(double x) { return (uint64_t)x; }
    __device__ static uint64_t unshift(double x, uint32_t s) { return (uint64_t)x >> s; }
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
    using Acc = uint64_t;
    static constexpr uint64_t sentinel() { return ~0ull; }
    __device__ static uint64_t from_u64(uint64_t x) { return x; }
    __device__ static uint64_t from_acc(uint64_t x) { return x; }
    __device__ static uint64_t val_to_u64(uint64_t x) { return x; }
    __device__ static uint64_t val_to_acc(uint64_t x) { return x; }
    __device__ static uint64_t unshift(uint64_t x, uint32_t s) { return x >> s; }
    __device__ static uint64_t add(uint64_t a, uint64_t b) { return a + b; }
    __device__ static uint64_t min(uint64_t a, uint64_t b) { return a < b ? a : b; }
    __device__ static void split(uint64_t key, uint32_t bits, uint32_t out_shift, uint64_t &val, uint32_t &c) {
        val = (key >> bits) << out_shift;
        c = (uint32_t)(key & ((1ull << bits) - 1));
    }
};

// 128-bit keys: cost * 2^bits + c for costs up to 2^64 (bits <= 16), so the
// packed key never overflows; table values are stored in 16 bytes.
using u128 = unsigned __int128;
template <> struct KeyOps<u128> {
    using Val = u128;
    using Acc = u128;
    static constexpr u128 sentinel() { return ~(u128)0; }
    __device__ static u128 from_acc(u128 x) { return x; }
    __device__ static uint64_t val_to_u64(u128 x) { return (uint64_t)x; }
    __device__ static u128 val_to_acc(u128 x) { return x; }
    __device__ static uint64_t unshift(u128 x, uint32_t s) { return (uint64_t)(x >> s); }
    __device__ static u128 add(u128 a, u128 b) { return a + b; }
    __device__ static u128 min(u128 a, u128 b) { return a < b ? a : b; }
    __device__ static void split(u128 key, uint32_t bits, uint32_t out_shift, u128 &val, uint32_t &c) {
        val = (key >> bits) << out_shift;
        c = (uint32_t)key & ((1u << bits) - 1u);
    }
};


// Buffer resource word 3 (data format 32-bit, raw addressing) for gfx9-family
// buffer instructions.
constexpr int kBufferWord3 = 0x00020000;

// ------------------------------------------------------------------ cost model (device)
// Layer cost t_l(v, c) = ceil(F / P) + r * (P_red - 1) * ceil(keep / (P / P_red)),
// with P the device count of the configuration and P_red the product of the
// split factors of the contracted dims.  With power-of-two factors (split rows
// hold exponents) the divisions are shifts; otherwise (rows hold the factors,
// P <= 255) they are integer divisions.  The host has bounded every operand so
// nothing overflows.
__device__ __forceinline__ uint64_t ceil_div_u64(uint64_t a, uint32_t b) { return (a + (b - 1)) / b; }

// Optional weight-gradient term: the weight tensor (weight_n words) is cut
// into shards of S = ceil(weight_n / P_w) words by the splits of its dims and
// each shard lives on the R = P / P_w devices that differ in the other dims;
// a ring all-reduce moves ceil(2 (R - 1) S / R) = 2S - floor(2S / R) words.
// Optional halo term: for every split loop dim k with a halo of width w, each
// part receives w boundary rows of the input from both neighbours along k; a
// row is the part's share of the input over its other dims:
// 2 w ceil(halo_n[k] / (product of the other input dims' splits)) words.
__device__ __forceinline__ uint64_t halo_cost(const DevVertex &dv, const uint8_t *ex, uint64_t r) {
    uint64_t words = 0;
    for (uint32_t k = 0; k < dv.ndims; k++) {
        if (!((dv.halo_mask >> k) & 1u) || ex[k] == (dv.factors ? 1 : 0)) continue;
        uint32_t S = dv.factors ? 1 : 0;
        for (uint32_t j = 0; j < dv.ndims; j++)
            if (j != k && ((dv.input_mask >> j) & 1u)) S = dv.factors ? S * ex[j] : S + ex[j];
        const uint64_t part = dv.factors ? ceil_div_u64(dv.halo_n[k], S)
                                         : (dv.halo_n[k] + ((1ull << S) - 1)) >> S;
        words += 2ull * dv.halo_w[k] * part;
    }
    return r * words;
}

__device__ __forceinline__ uint64_t layer_cost(const DevVertex &dv, const uint8_t *ex, uint64_t r) {
    const uint64_t halo = dv.halo_mask ? halo_cost(dv, ex, r) : 0;
    if (dv.factors) {
        uint32_t P = 1, red = 1, Pw = 1;
        for (uint32_t k = 0; k < dv.ndims; k++) {
            P *= ex[k];
            if ((dv.reduce_mask >> k) & 1u) red *= ex[k];
            if ((dv.weight_mask >> k) & 1u) Pw *= ex[k];
        }
        uint64_t cost = ceil_div_u64(dv.flops, P) + r * ((uint64_t)(red - 1) * ceil_div_u64(dv.keep_n, P / red));
        if (dv.weight_n) {
            const uint64_t S2 = 2 * ceil_div_u64(dv.weight_n, Pw);
            cost += r * (S2 - S2 / (P / Pw));
        }
        return cost + halo;
    }
    uint32_t E = 0, ered = 0, ew = 0;
    for (uint32_t k = 0; k < dv.ndims; k++) {
        E += ex[k];
        if ((dv.reduce_mask >> k) & 1u) ered += ex[k];
        if ((dv.weight_mask >> k) & 1u) ew += ex[k];
    }
    uint64_t compute = (dv.flops + ((1ull << E) - 1)) >> E;
    uint32_t ek = E - ered;
    uint64_t part = (dv.keep_n + ((1ull << ek) - 1)) >> ek;
    uint64_t cost = compute + r * (((1ull << ered) - 1) * part);
    if (dv.weight_n) {
        const uint64_t S2 = 2 * ((dv.weight_n + ((1ull << ew) - 1)) >> ew);
        cost += r * (S2 - (S2 >> (E - ew)));
    }
    return cost + halo;
}

// Device byte of one configuration: the exponent sum log2(P) of power-of-two
// rows, else the device count P itself.
__device__ __forceinline__ uint32_t device_byte(const DevVertex &dv, const uint8_t *ex) {
    uint32_t x = dv.factors ? 1 : 0;
    for (uint32_t k = 0; k < dv.ndims; k++) x = dv.factors ? x * ex[k] : x + ex[k];
    return x;
}

// Split signature of one endpoint configuration of an edge: the split of every
// tensor dim (an unsplit dim counts as factor 1), one field per dim -- 5-bit
// exponents, or 8-bit factors.  Two endpoints redistribute nothing exactly when
// their signatures are equal.
__device__ __forceinline__ uint64_t split_signature(const int8_t *dims, uint32_t rank, const uint8_t *ex,
                                                   uint32_t factors) {
    const uint32_t w = factors ? 8 : 5, one = factors ? 1 : 0;
    uint64_t sig = 0;
    for (uint32_t k = 0; k < rank; k++) sig |= (uint64_t)(dims[k] >= 0 ? ex[dims[k]] : one) << (w * k);
    return sig;
}

// r * t_x of the volume-intersection model for one (producer config, consumer
// config) pair.  Device d of a configuration is the mixed-radix point of its
// split grid (loop dim 0 slowest); a tensor dim is cut into equal fractions on
// each side by the split of the loop dim it maps to (1 if unmapped).  Per
// tensor dim the parts of u and v are measured in units of 1/(s_u * s_v):
// v's part [x_v * s_u, (x_v + 1) * s_u), u's part [x_u * s_v, (x_u + 1) * s_v).
// forward  = max_d |need_v(d)| - |need_v(d) n hold_u(d)|, backward the same with
// u and v swapped; words = ceil(elems * fraction) per direction.  The host
// checks Q = prod s_u * s_v < 2^32, so every endpoint and volume in units fits
// 32 bits.  Devices that only one side uses contribute that side's whole part
// (a constant), so the walk covers the devices both use, as odometers over
// the two grids, and stops once both maxima reach their ceilings.
__device__ __forceinline__ uint64_t ceil_frac(uint64_t elems, uint64_t f, uint64_t Q) {
    // elems * f / Q rounded up, f <= Q < 2^32: (elems % Q) * f < Q^2 < 2^64
    const uint64_t q = elems / Q, rem = elems % Q;
    return q * f + (rem * f + Q - 1) / Q;
}

__device__ __forceinline__ uint32_t split_of(const DevVertex &x, const uint8_t *ex, int k) {
    return x.factors ? ex[k] : 1u << ex[k];
}

// With m = min over the devices both ends use of |need_v(d) n hold_u(d)|:
// forward = need_v - m (need_v when v uses more devices), backward = hold_u - m
// (hold_u when u uses more).  Per tensor dim the device's coordinate on each
// side advances every `stride` devices (the product of the splits of the loop
// dims after the mapped one) and wraps at the split; all per-dim state is
// indexed by unrolled constants so it stays in registers.
//
// Power-of-two splits take the closed form of k_edge_volume_pow2 instead.
__device__ __forceinline__ uint64_t volume_cost(const DevVertex &u, const uint8_t *exu, const DevVertex &v,
                                                const uint8_t *exv, const DevEdge &de, uint64_t r) {
    uint32_t Pu = 1, Pv = 1;
    for (uint32_t k = 0; k < u.ndims; k++) Pu *= split_of(u, exu, (int)k);
    for (uint32_t k = 0; k < v.ndims; k++) Pv *= split_of(v, exv, (int)k);
    uint32_t ta[kMaxDims], tb[kMaxDims], stu[kMaxDims], stv[kMaxDims];
    uint32_t xu[kMaxDims], xv[kMaxDims], pu[kMaxDims], pv[kMaxDims];
    uint32_t Q = 1, need_v = 1, hold_u = 1;
#pragma unroll
    for (int t = 0; t < kMaxDims; t++) {
        ta[t] = tb[t] = stu[t] = stv[t] = 1;
        xu[t] = xv[t] = pu[t] = pv[t] = 0;
        if (t < (int)de.rank) {
            const int ka = de.sdim[t], kb = de.ddim[t];
            if (ka >= 0) {
                ta[t] = split_of(u, exu, ka);
                for (int k = ka + 1; k < (int)u.ndims; k++) stu[t] *= split_of(u, exu, k);
            }
            if (kb >= 0) {
                tb[t] = split_of(v, exv, kb);
                for (int k = kb + 1; k < (int)v.ndims; k++) stv[t] *= split_of(v, exv, k);
            }
            Q *= ta[t] * tb[t];
            need_v *= ta[t];      // |v's part| = 1/b = a units
            hold_u *= tb[t];
        }
    }
    const uint32_t both = Pu < Pv ? Pu : Pv;
    uint32_t m = need_v < hold_u ? need_v : hold_u;
    for (uint32_t d = 0; d < both && m; d++) {
        uint32_t common = 1;
#pragma unroll
        for (int t = 0; t < kMaxDims; t++) {
            if (t < (int)de.rank) {
                const uint32_t a = ta[t], b = tb[t], cu = xu[t], cv = xv[t];
                const uint32_t lo = cv * a > cu * b ? cv * a : cu * b;
                const uint32_t hi = (cv + 1) * a < (cu + 1) * b ? (cv + 1) * a : (cu + 1) * b;
                common *= hi > lo ? hi - lo : 0;
                // next device
                if (++pu[t] == stu[t]) { pu[t] = 0; if (++xu[t] == ta[t]) xu[t] = 0; }
                if (++pv[t] == stv[t]) { pv[t] = 0; if (++xv[t] == tb[t]) xv[t] = 0; }
            }
        }
        m = common < m ? common : m;
    }
    const uint32_t fwd = Pv > Pu ? need_v : need_v - m, bwd = Pu > Pv ? hold_u : hold_u - m;
    return r * (ceil_frac(de.elems, fwd, Q) + ceil_frac(de.elems, bwd, Q));
}

// r * t_x from the two signatures and device bytes of the endpoints.
__device__ __forceinline__ uint64_t edge_cost_sig(uint64_t sig_a, uint64_t sig_b, uint32_t la, uint32_t lb,
                                                  uint64_t elems, uint64_t r, uint32_t factors) {
    if (sig_a == sig_b) return 0;
    uint32_t s = la > lb ? la : lb;
    if (factors) return r * ceil_div_u64(elems, s);
    return r * ((elems + ((1ull << s) - 1)) >> s);
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

// The small vertices of the bulk lane schedule (the chains of dependent
// vertices) run their waves at the highest issue priority: on a SIMD shared
// with the long fills of the bulk stream they then issue first.
__device__ __forceinline__ void set_priority(const BatchEntry &e) {
    if (e.prio) __builtin_amdgcn_s_setprio(3);
}

// The key of configuration c of vertex `me` under plan digits dv, summed over
// contributions [c0, c1): plain costs (layer, transfer) are summed in `sum`
// and shifted into key space at the end; DP tables are stored in this
// vertex's key space already; the layer term carries c into the low bits.
template <typename KeyT>
__device__ __forceinline__ typename KeyOps<KeyT>::Acc contrib_key(const Contrib *__restrict__ cb, uint32_t c0, uint32_t c1,
                                                const DevVertex &me, uint32_t c, const uint32_t (&dv)[kMaxDep],
                                                uint32_t bits, const DevVertex *__restrict__ V,
                                                const DevEdge *__restrict__ E, const uint64_t *__restrict__ L,
                                                const uint8_t *__restrict__ lsum, const uint64_t *__restrict__ sig,
                                                uint64_t r) {
    using Val = typename KeyOps<KeyT>::Val;
    using Acc = typename KeyOps<KeyT>::Acc;
    uint64_t sum = 0, low = 0;
    Acc keysum = 0;
    for (uint32_t k = c0; k < c1; k++) {
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
            sum += edge_cost_sig(sme, sot, lsum[me.L_off + c], lsum[ov.L_off + xo], de.elems, r, de.factors);
        } else {
            uint64_t idx = (uint64_t)c * ct.sc;
            for (int k2 = 0; k2 < kMaxDep; k2++) idx += (uint64_t)dv[k2] * ct.sd[k2];
            if (ct.raw_u64) sum += ((const uint64_t *)ct.ptr)[idx];
            else keysum += KeyOps<KeyT>::val_to_acc(((const Val *)ct.ptr)[idx]);
        }
    }
    return ((Acc)sum << bits) + keysum + low;
}

// One workgroup handles `span` runs of kPrepThreads consecutive (c, column)
// elements of one outer index of one block, so the block, its contributions
// and the outer digits are uniform across the workgroup (scalar loads, which
// later runs find in the scalar cache); lanes differ only in (c, column).
template <typename KeyT>
__device__ __forceinline__ void prep_item(const PrepArgs &a, uint32_t wg, const DevVertex *__restrict__ V,
                                          const DevEdge *__restrict__ E, const uint64_t *__restrict__ L,
                                          const uint8_t *__restrict__ lsum, const uint64_t *__restrict__ sig,
                                          const Contrib *__restrict__ cb, uint64_t r) {
    KeyT *__restrict__ blocks = (KeyT *)a.blocks;
    uint32_t b = 0;
    while (b + 1 < a.nblocks && wg >= a.blk[b + 1].wg_begin) b++;
    b = __builtin_amdgcn_readfirstlane(b);
    const Block &bk = a.blk[b];
    const uint32_t rel = wg - bk.wg_begin;
    const uint32_t row = rel / bk.chunks, chunk = rel % bk.chunks;
    const uint32_t per_row = a.K * bk.ld;
    uint32_t dv[kMaxDep];
    for (int k = 0; k < kMaxDep; k++) dv[k] = 0;
    uint32_t x = row;
    for (int k = (int)bk.npre - 1; k >= 0; k--) {
        dv[bk.pre[k]] = x % bk.prerad[k];
        x /= bk.prerad[k];
    }
    const DevVertex me = V[a.vi];
    for (uint32_t s = 0; s < bk.span; s++) {
        const uint32_t e = (chunk * bk.span + s) * kPrepThreads + threadIdx.x;
        if (e >= per_row) return;
        const uint32_t c = e / bk.ld, q = e % bk.ld;
        KeyT *out = blocks + bk.out_off + (uint64_t)row * per_row + e;
        if (bk.post >= 0 && q >= bk.postrad) {
            *out = (KeyT)0;
            continue;
        }
        if (bk.post >= 0) dv[bk.post] = q;
        *out = KeyOps<KeyT>::from_acc(contrib_key<KeyT>(cb, bk.c_begin, bk.c_end, me, c, dv, a.bits, V, E, L,
                                                         lsum, sig, r));
    }
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

template <typename KeyT>
using MergeBuf = KeyT[2][kMergeVals][64];

// Workgroup b of one vertex's row fill; xch: the workgroup's LDS merge buffer.
template <typename KeyT, int TZ, int TM, int NA>
__device__ __forceinline__ void rows_item(const RowsArgs &a, uint32_t b, MergeBuf<KeyT> &xch) {
    using Ops = KeyOps<KeyT>;
    using Val = typename Ops::Val;
    const uint32_t lane = threadIdx.x & 63;
    // the wave index is uniform across the wave: say so, so that everything
    // derived from it (c range, column addresses) lives in SGPRs
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // blocks are dealt round-robin to the 8 XCDs: give every XCD a contiguous
    // range of tiles so that tiles sharing a column slice share an L2 (every
    // vertex's block count and first block are multiples of 8, so the XCD of
    // a block is its local index mod 8)
    const uint32_t nb = a.nblocks_launched;
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
    // keep U = 4 values in flight per set; 8-column tiles keep 2 (two sets of
    // 2 x 8 keys still fit in SGPRs) -- they serve the small, latency-bound
    // vertices, whose waves otherwise wait out a round trip per c.  Loads past
    // c1 repeat column c1 - 1 (in bounds, unused) so that every load is
    // unconditional and the register sets never need copying.
    constexpr int U = TZ <= 2 ? 4 : TZ <= 8 ? 2 : 1;
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
    // fused minimum of the reader v_j (c_j = z): per row, its keys over this
    // tile's columns -- the stored value of T[z][r] (already in v_j's key
    // space) plus v_j's other row terms at (r, z) and its column block at z
    // -- reduced in the lane, then min-combined across tiles atomically
    constexpr bool kFuse = sizeof(KeyT) == 8;
    const bool fuse = kFuse && a.fz_keys != nullptr;
#pragma unroll
    for (int m = 0; m < TM; m++) {
        if (!valid[m]) continue;
        const uint64_t base_idx = (uint64_t)o * a.MR + r[m];
        uint32_t fzoff[kMaxATerms];
        KeyT best = Ops::sentinel();
        if (fuse) {
            uint32_t x = r[m], dR[kMaxDep];
            for (int k = kMaxDep - 1; k >= 0; k--)
                if (k < (int)a.nR) { dR[k] = x % a.radR[k]; x /= a.radR[k]; } else dR[k] = 0;
            for (int q = 0; q < kMaxATerms; q++) {
                uint32_t off = 0;
                if (q < (int)a.fz_na)
                    for (int k = 0; k < kMaxDep; k++) off += dR[k] * a.fz_a[q].sdR[k];
                fzoff[q] = off;
            }
        }
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
                    if (a.T) ((Val *)a.T)[idx] = v;
                    a.A[idx] = (uint16_t)cc;
                    if constexpr (kFuse) {
                        if (fuse) {
                            KeyT k = __builtin_bit_cast(KeyT, v);
                            for (int q = 0; q < kMaxATerms; q++)
                                if (q < (int)a.fz_na)
                                    k = Ops::add(k, ((const KeyT *)a.fz_a[q].ptr)[fzoff[q] + z * a.fz_a[q].sc]);
                            k = Ops::add(k, ((const KeyT *)a.fz_B)[(uint64_t)z * a.fz_ldz]);
                            best = Ops::min(best, k);
                        }
                    }
                }
            }
        }
        if constexpr (kFuse) {
            if (fuse)
                atomicMin((unsigned long long *)a.fz_keys + r[m],
                          (unsigned long long)__builtin_bit_cast(uint64_t, best));
        }
    }
}

template <typename KeyT>
__device__ __forceinline__ void reduce_item(const ReduceArgs &a, uint32_t lb) {
    using Ops = KeyOps<KeyT>;
    using Val = typename Ops::Val;
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
    constexpr int W = sizeof(KeyT) / 4;   // 32-bit words of a key
    struct Words { uint32_t w[W]; };
    Words x = __builtin_bit_cast(Words, v);
#pragma unroll
    for (int k = 0; k < W; k++) x.w[k] = (uint32_t)__shfl_xor((int)x.w[k], mask, 64);
    return __builtin_bit_cast(KeyT, x);
}

template <typename KeyT, int NT>
__device__ __forceinline__ void generic_item(const GenericArgs &a, uint32_t lb) {
    using Ops = KeyOps<KeyT>;
    using Val = typename Ops::Val;
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

// ------------------------------------------------------------------ direct fill (small vertices)
// Like the generic fill, 2^group_log2 lanes share one table entry and stride
// over c.  Each lane first resolves every contribution for its entry once --
// an array read at base + c * stride (layer costs, caller or volume edge
// matrices, producer tables) or a split-signature edge term with the other
// endpoint's signature and device byte fixed -- so the loop over c only loads
// data.  Vertices with more contributions than fit the register set take the
// per-cell path of the prep kernel.
constexpr int kDirectTerms = 8;

template <typename KeyT>
__device__ __forceinline__ void direct_item(const DirectArgs &a, uint32_t lb, const DevVertex *__restrict__ V,
                                            const DevEdge *__restrict__ E, const uint64_t *__restrict__ L,
                                            const uint8_t *__restrict__ lsum, const uint64_t *__restrict__ sig,
                                            const Contrib *__restrict__ cb, uint64_t r, KeyT (&xch)[4]) {
    using Ops = KeyOps<KeyT>;
    using Val = typename Ops::Val;
    const uint32_t G = 1u << a.group_log2;
    const uint64_t nthreads = (uint64_t)a.N << a.group_log2;
    const DevVertex me = V[a.vi];
    const uint32_t nt = a.c_end - a.c_begin;
    const bool fast = nt <= (uint32_t)kDirectTerms;
    for (uint64_t tid = lb * (uint64_t)blockDim.x + threadIdx.x; tid < ((nthreads + 255) / 256) * 256;
         tid += (uint64_t)a.nblk * blockDim.x) {
        const bool live = tid < nthreads;
        const uint64_t phi = live ? tid >> a.group_log2 : a.N - 1;
        const uint32_t lane = (uint32_t)(tid & (G - 1));
        uint32_t dv[kMaxDep];
        uint64_t x = phi;
        for (int k = kMaxDep - 1; k >= 0; k--)
            if (k < (int)a.m) { dv[k] = (uint32_t)(x % a.rad[k]); x /= a.rad[k]; } else dv[k] = 0;
        KeyT best = Ops::sentinel();
        if (fast) {
            // kind: 0 plain u64 array, 1 key-space table, 2 signature edge
            const char *base[kDirectTerms];
            uint32_t stride[kDirectTerms], kind[kDirectTerms], lot[kDirectTerms], fac[kDirectTerms];
            const uint8_t *lme[kDirectTerms];
            uint64_t sot[kDirectTerms], elems[kDirectTerms];
#pragma unroll
            for (int t = 0; t < kDirectTerms; t++) {
                base[t] = nullptr;
                lme[t] = nullptr;
                stride[t] = kind[t] = lot[t] = fac[t] = 0;
                sot[t] = elems[t] = 0;
                if (t < (int)nt) {
                    const Contrib ct = cb[a.c_begin + t];
                    if (ct.kind == kContribLayer) {
                        base[t] = (const char *)(L + me.L_off);
                        stride[t] = 8;
                    } else if (ct.kind == kContribEdge) {
                        const DevEdge de = E[ct.edge];
                        const uint32_t xo = dv[ct.dig];
                        const DevVertex ov = V[ct.vi_is_src ? de.dst : de.src];
                        kind[t] = 2;
                        base[t] = (const char *)(sig + de.sig_off + (ct.vi_is_src ? 0 : V[de.src].K));
                        stride[t] = 8;
                        sot[t] = sig[de.sig_off + (ct.vi_is_src ? me.K : 0) + xo];
                        lme[t] = lsum + me.L_off;
                        lot[t] = lsum[ov.L_off + xo];
                        elems[t] = de.elems;
                        fac[t] = de.factors;
                    } else {
                        uint64_t idx = 0;
                        for (int k2 = 0; k2 < kMaxDep; k2++) idx += (uint64_t)dv[k2] * ct.sd[k2];
                        kind[t] = ct.raw_u64 ? 0 : 1;
                        stride[t] = ct.sc * 8;
                        base[t] = (const char *)ct.ptr + idx * 8;
                    }
                }
            }
            for (uint32_t c = lane; c < a.K; c += G) {
                uint64_t sum = 0, keysum = 0;
#pragma unroll
                for (int t = 0; t < kDirectTerms; t++) {
                    if (t < (int)nt) {
                        if (kind[t] == 2) {
                            const uint64_t sme = *(const uint64_t *)(base[t] + (uint64_t)c * stride[t]);
                            sum += edge_cost_sig(sme, sot[t], lme[t][c], lot[t], elems[t], r, fac[t]);
                        } else {
                            const uint64_t v = *(const uint64_t *)(base[t] + (uint64_t)c * stride[t]);
                            if (kind[t] == 0) sum += v;
                            else keysum += Ops::val_to_u64(__builtin_bit_cast(Val, v));
                        }
                    }
                }
                // the layer term is always present: c fills the low bits
                best = Ops::min(best, Ops::from_u64((sum << a.bits) + keysum + c));
            }
        } else {
            for (uint32_t c = lane; c < a.K; c += G)
                best = Ops::min(best, Ops::from_acc(contrib_key<KeyT>(cb, a.c_begin, a.c_end, me, c, dv, a.bits, V,
                                                                      E, L, lsum, sig, r)));
        }
        for (uint32_t m = (G < 64 ? G : 64) >> 1; m > 0; m >>= 1) best = Ops::min(best, shfl_xor_key(best, (int)m));
        if (G > 64) {
            // a group of 2 or 4 waves: their minima meet in LDS (every thread
            // of the workgroup runs the same iterations, so the barriers match)
            const uint32_t wave = threadIdx.x >> 6;
            if ((threadIdx.x & 63) == 0) xch[wave] = best;
            __syncthreads();
            if (lane == 0)
                for (uint32_t w = 1; w < G / 64; w++) best = Ops::min(best, xch[wave + w]);
            __syncthreads();
        }
        if (live && lane == 0) {
            Val v;
            uint32_t cc;
            Ops::split(best, a.bits, a.out_shift, v, cc);
            ((Val *)a.T)[phi] = v;
            a.A[phi] = (uint16_t)cc;
        }
    }
}

}  // namespace pase
