/*
 * Plain CPU oracle for PaSE's strategy search (Elango, "PaSE: Parallelization
 * Strategies for Efficient DNN Training", IPDPS 2021).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this file's library.  It shares no
 * code with the HIP library and is deliberately slow and literal:
 *
 *   - configurations: Sec. II, C(v) = {c : prod c_k <= p}, either every tuple
 *     of positive integers (oracle_configs_all) or only powers of two
 *     (oracle_configs, p = 2^L), enumerated in lexicographic order of the
 *     split tuple (first loop dim slowest);
 *   - cost function F: eq. (1), with the integer layer / transfer cost model
 *     documented at layer_cost() and transfer_cost();
 *   - vertex ordering: GenerateSeq, Fig. 3 (argmin of |u.d|, ties to the
 *     lowest vertex id);
 *   - dynamic program: recurrence (4) evaluated as in FindBestStrategy, Fig. 4,
 *     with the node function of eq. (3), the connected set X(i) and connected
 *     subsets S(i) of Sec. III-B, the strict "<" update over configurations in
 *     ascending index order, and back-substitution from the last vertex;
 *   - device assignment after the search: the greedy locality-maximising
 *     placement of Sec. II's device-assignment paragraph (oracle_assign_devices),
 *     repeated argmax over every (part, device) pair, shared elements counted
 *     cell by cell;
 *   - every addition is overflow-checked in uint64.
 *
 * Tables are stored in canonical order: the dependent set D(i) sorted by
 * vertex id, first digit slowest.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <stdio.h>
#include <time.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define MAXD 8

typedef struct {
    /* graph */
    int nv, ne;
    int ndims[4096];
    uint64_t *size;          /* nv*MAXD */
    uint32_t *reduce_mask;   /* nv */
    uint64_t *fpp;           /* nv flops per iteration point */
    int *src, *dst, *rank;   /* ne */
    int *src_dim, *dst_dim;  /* ne*MAXD */
    uint64_t *elems;         /* ne */
    uint64_t r;              /* FLOP-to-byte ratio weighting communication */
    int xmodel;              /* transfer cost: 0 split match, 1 volume intersection */
    int grad_sync;           /* 1: layer cost adds the weight-gradient all-reduce */
    uint32_t *weight_mask;   /* nv: loop dims indexing the layer's weights (0: none) */
    uint64_t *wpp;           /* nv: weight words per point of those dims */
    int halo_model;          /* 1: layer cost adds the halo exchange of convolutions */
    uint32_t *halo;          /* nv*MAXD: halo width of each loop dim (0: none) */
    uint32_t *in_mask;       /* nv: loop dims indexing the layer's input tensor */
    /* configurations */
    int p;
    int *K;                  /* configs per vertex */
    uint32_t **sp;           /* sp[v][c*ndims+k] = split factor of dim k */
    /* cost tables */
    uint64_t **Lc;           /* Lc[v][c]       = t_l(v, c)            */
    uint64_t **Rx;           /* Rx[e][cu*Kv+cv] = r * t_x(e, cu, cv)  */
    /* undirected neighbourhoods, deduplicated: nbr[v][0..deg[v]) */
    int **nbr, *deg;
    /* ordering */
    int *seq, *pos;          /* seq[i] = vertex at position i, pos[v] = its position */
    int **D, *nD;            /* D[i] = dependent set of position i, sorted by vertex id */
    /* DP tables by position */
    uint64_t *N;             /* entries of table i */
    uint64_t **T;            /* cost tables */
    uint16_t **A;            /* argmin tables (config index of seq[i]) */
    uint64_t min_cost;
    int *strategy;           /* config index per vertex id */
    int solved;
    uint64_t cells, cells_done;
    double seconds;
    int overflow;
    char err[256];
} oracle_t;

static int fail(oracle_t *o, const char *msg) {
    snprintf(o->err, sizeof o->err, "%s", msg);
    return 1;
}

const char *oracle_error(oracle_t *o) { return o->err; }

static int add_ok(uint64_t a, uint64_t b, uint64_t *out) { return !__builtin_add_overflow(a, b, out); }
static int mul_ok(uint64_t a, uint64_t b, uint64_t *out) { return !__builtin_mul_overflow(a, b, out); }

static uint64_t ceil_div(uint64_t a, uint64_t b) { return a / b + (a % b != 0); }

/* ------------------------------------------------------------------ graph */

oracle_t *oracle_new(int nv, const int *ndims, const uint64_t *sizes, const uint32_t *reduce_mask,
                     const uint64_t *fpp, int ne, const int *src, const int *dst, const int *rank,
                     const int *src_dim, const int *dst_dim, const uint64_t *elems, uint64_t r) {
    if (nv < 1 || nv > 4096 || ne < 0) return NULL;
    oracle_t *o = calloc(1, sizeof *o);
    o->nv = nv; o->ne = ne; o->r = r;
    o->size = calloc((size_t)nv * MAXD, sizeof(uint64_t));
    o->reduce_mask = calloc(nv, sizeof(uint32_t));
    o->fpp = calloc(nv, sizeof(uint64_t));
    o->weight_mask = calloc(nv, sizeof(uint32_t));
    o->wpp = calloc(nv, sizeof(uint64_t));
    o->halo = calloc((size_t)nv * MAXD, sizeof(uint32_t));
    o->in_mask = calloc(nv, sizeof(uint32_t));
    for (int v = 0; v < nv; v++) {
        o->ndims[v] = ndims[v];
        for (int k = 0; k < ndims[v]; k++) o->size[v * MAXD + k] = sizes[v * MAXD + k];
        o->reduce_mask[v] = reduce_mask[v];
        o->fpp[v] = fpp[v];
    }
    o->src = calloc(ne + 1, sizeof(int)); o->dst = calloc(ne + 1, sizeof(int));
    o->rank = calloc(ne + 1, sizeof(int));
    o->src_dim = calloc((size_t)(ne + 1) * MAXD, sizeof(int));
    o->dst_dim = calloc((size_t)(ne + 1) * MAXD, sizeof(int));
    o->elems = calloc(ne + 1, sizeof(uint64_t));
    for (int e = 0; e < ne; e++) {
        o->src[e] = src[e]; o->dst[e] = dst[e]; o->rank[e] = rank[e]; o->elems[e] = elems[e];
        for (int k = 0; k < rank[e]; k++) {
            o->src_dim[e * MAXD + k] = src_dim[e * MAXD + k];
            o->dst_dim[e * MAXD + k] = dst_dim[e * MAXD + k];
        }
    }
    /* N(v) = {u : (u,v) in E or (v,u) in E}, as a set (Sec. III notation) */
    o->deg = calloc(nv, sizeof(int));
    o->nbr = calloc(nv, sizeof(int *));
    char *adj = calloc((size_t)nv * nv, 1);
    for (int e = 0; e < ne; e++) {
        adj[(size_t)src[e] * nv + dst[e]] = 1;
        adj[(size_t)dst[e] * nv + src[e]] = 1;
    }
    for (int v = 0; v < nv; v++) {
        o->nbr[v] = calloc(nv, sizeof(int));
        for (int u = 0; u < nv; u++)
            if (adj[(size_t)v * nv + u]) o->nbr[v][o->deg[v]++] = u;
    }
    free(adj);
    return o;
}

static void free_tables(oracle_t *o) {
    if (o->T) {
        for (int i = 0; i < o->nv; i++) { free(o->T[i]); free(o->A[i]); free(o->D[i]); }
        free(o->T); free(o->A); free(o->D); free(o->nD); free(o->N);
        free(o->seq); free(o->pos); free(o->strategy);
        o->T = NULL;
    }
}

static void free_configs(oracle_t *o) {
    if (o->K) {
        for (int v = 0; v < o->nv; v++) { free(o->sp[v]); free(o->Lc[v]); }
        for (int e = 0; e < o->ne; e++) free(o->Rx[e]);
        free(o->sp); free(o->Lc); free(o->Rx); free(o->K);
        o->K = NULL;
    }
}

void oracle_free(oracle_t *o) {
    if (!o) return;
    free_tables(o);
    free_configs(o);
    for (int v = 0; v < o->nv; v++) free(o->nbr[v]);
    free(o->nbr); free(o->deg);
    free(o->size); free(o->reduce_mask); free(o->fpp); free(o->weight_mask); free(o->wpp);
    free(o->halo); free(o->in_mask);
    free(o->src); free(o->dst); free(o->rank); free(o->src_dim); free(o->dst_dim); free(o->elems);
    free(o);
}

/* --------------------------------------------------------- configurations */

/* Append every split tuple of dims k..d-1 in lexicographic order (dim 0
 * slowest): with `pow2`, the powers of two with product <= budget, else every
 * positive integer tuple with product <= budget (out = NULL: count only).
 * Returns 0 when more than `cap` tuples would be produced. */
static int enum_rec(int d, int k, uint64_t budget, int pow2, uint32_t *cur, uint32_t *out, int *count, int cap) {
    if (k == d) {
        if (*count >= cap) return 0;
        if (out) memcpy(out + (size_t)(*count) * d, cur, d * sizeof(uint32_t));
        (*count)++;
        return 1;
    }
    for (uint64_t s = 1; s <= budget; s = pow2 ? 2 * s : s + 1) {
        cur[k] = (uint32_t)s;
        if (!enum_rec(d, k + 1, budget / s, pow2, cur, out, count, cap)) return 0;
    }
    return 1;
}

/* Layer cost t_l(v, c): compute time plus r times the intra-layer
 * communication (eq. 1 and the text after it).  Integer model:
 *   compute = ceil(fpp * prod(n_k) / P),  P = prod(s_k)
 *   comm    = (prod_{k in reduce} s_k - 1) * ceil(prod_{k not in reduce} n_k
 *                                                 / prod_{k not in reduce} s_k)
 *   t_l     = compute + r * comm
 * (comm is the partial-sum reduction a split contraction dim requires.)
 * With grad_sync, t_l also carries the data-parallel weight-gradient
 * all-reduce (an assumed form, as the paper prints no formula; see
 * oracle_set_grad_sync); with the halo model, the halo exchange of a
 * convolution (oracle_set_halo_model). */
static int layer_cost(oracle_t *o, int v, const uint32_t *s, uint64_t *out) {
    uint64_t flops = o->fpp[v], P = 1, red_split = 1, keep_n = 1, keep_split = 1;
    for (int k = 0; k < o->ndims[v]; k++) {
        uint64_t n = o->size[v * MAXD + k];
        if (!mul_ok(flops, n, &flops)) return 0;
        P *= s[k];
        if (o->reduce_mask[v] >> k & 1u) {
            red_split *= s[k];
        } else {
            if (!mul_ok(keep_n, n, &keep_n)) return 0;
            keep_split *= s[k];
        }
    }
    uint64_t compute = ceil_div(flops, P);
    uint64_t comm, comm_r, total;
    if (!mul_ok(red_split - 1, ceil_div(keep_n, keep_split), &comm)) return 0;
    if (!mul_ok(o->r, comm, &comm_r)) return 0;
    if (!add_ok(compute, comm_r, &total)) return 0;
    if (o->grad_sync && o->weight_mask[v]) {
        /* the weight tensor (wpp words per point of the weight dims) is cut by
         * the splits of the weight dims into shards of S words; each shard is
         * held by the R devices that differ only in the other dims, which
         * all-reduce its gradient: a ring moves 2 (R - 1) / R * S words per
         * device */
        uint64_t W = o->wpp[v], Pw = 1, R = 1;
        for (int k = 0; k < o->ndims[v]; k++) {
            if (o->weight_mask[v] >> k & 1u) {
                if (!mul_ok(W, o->size[v * MAXD + k], &W)) return 0;
                Pw *= s[k];
            } else {
                R *= s[k];
            }
        }
        uint64_t S = ceil_div(W, Pw);
        unsigned __int128 words = ((unsigned __int128)2 * (R - 1) * S + (R - 1)) / R;
        uint64_t grad;
        if (words >> 64 || !mul_ok(o->r, (uint64_t)words, &grad) || !add_ok(total, grad, &total)) return 0;
    }
    if (o->halo_model) {
        /* a part along loop dim k (halo width w, the kernel's half extent
         * along an input spatial dim) needs w boundary rows of the input from
         * each of its two neighbours once dim k is split; a row spans the
         * part's share of the input tensor over its other dims */
        for (int k = 0; k < o->ndims[v]; k++) {
            uint64_t w = o->halo[v * MAXD + k];
            if (w == 0 || s[k] == 1) continue;
            uint64_t rest = 1, rest_split = 1, words, cost;
            for (int j = 0; j < o->ndims[v]; j++) {
                if (j == k || !(o->in_mask[v] >> j & 1u)) continue;
                if (!mul_ok(rest, o->size[v * MAXD + j], &rest)) return 0;
                rest_split *= s[j];
            }
            if (!mul_ok(2 * w, ceil_div(rest, rest_split), &words)) return 0;
            if (!mul_ok(o->r, words, &cost) || !add_ok(total, cost, &total)) return 0;
        }
    }
    *out = total;
    return 1;
}

/* Convolution geometry of the layers: halo[v*MAXD+k] = halo width of loop dim
 * k of v (0: none), in_mask[v] = loop dims indexing v's input tensor.  Used by
 * the halo term. */
int oracle_set_halo(oracle_t *o, const uint32_t *halo, const uint32_t *in_mask) {
    for (int v = 0; v < o->nv; v++) {
        if (in_mask[v] >> o->ndims[v]) return fail(o, "input dim out of range");
        for (int k = 0; k < MAXD; k++) {
            uint32_t w = halo[v * MAXD + k];
            if (w && (k >= o->ndims[v] || !(in_mask[v] >> k & 1u))) return fail(o, "halo on a non-input dim");
            o->halo[v * MAXD + k] = w;
        }
        o->in_mask[v] = in_mask[v];
    }
    return 0;
}

/* 1: the next configuration enumeration adds the halo exchange of
 * convolutions to every layer cost.  The paper lists halo communication among
 * the intra-layer communication of t_l without printing a formula; this
 * oracle takes the exchange of w rows with both neighbours along each split
 * halo dim, in words per device. */
int oracle_set_halo_model(oracle_t *o, int on) {
    o->halo_model = on != 0;
    return 0;
}

/* Weight tensors of the layers: mask[v] = loop dims indexing v's weights,
 * wpp[v] = words per point of those dims.  Used by the gradient term. */
int oracle_set_weights(oracle_t *o, const uint32_t *mask, const uint64_t *wpp) {
    for (int v = 0; v < o->nv; v++) {
        if (mask[v] >> o->ndims[v]) return fail(o, "weight dim out of range");
        o->weight_mask[v] = mask[v];
        o->wpp[v] = wpp[v];
    }
    return 0;
}

/* 1: the next configuration enumeration adds the weight-gradient all-reduce
 * to every layer cost.  Data parallelism replicates weights, and Sec. I names
 * the gradient all-reduce as its communication, but no formula is printed;
 * this oracle takes a ring all-reduce of each weight shard among its replicas. */
int oracle_set_grad_sync(oracle_t *o, int on) {
    o->grad_sync = on != 0;
    return 0;
}

/* r * t_x(u, v): zero when both endpoints split every dim of the tensor the
 * same way, otherwise the tensor is re-distributed: ceil(elems / max(P_u, P_v))
 * words per device, weighted by r.  Symmetric in (u, v) as the paper requires. */
static int transfer_cost(oracle_t *o, int e, const uint32_t *su_, const uint32_t *sv_, uint64_t *out) {
    int u = o->src[e], v = o->dst[e];
    int match = 1;
    for (int k = 0; k < o->rank[e]; k++) {
        int a = o->src_dim[e * MAXD + k], b = o->dst_dim[e * MAXD + k];
        uint64_t su = a >= 0 ? su_[a] : 1;
        uint64_t sv = b >= 0 ? sv_[b] : 1;
        if (su != sv) match = 0;
    }
    if (match) { *out = 0; return 1; }
    uint64_t Pu = 1, Pv = 1;
    for (int k = 0; k < o->ndims[u]; k++) Pu *= su_[k];
    for (int k = 0; k < o->ndims[v]; k++) Pv *= sv_[k];
    uint64_t words = ceil_div(o->elems[e], Pu > Pv ? Pu : Pv);
    return mul_ok(o->r, words, out);
}

/* Volume-intersection transfer cost (Sec. II).  A(v,d) is the part of the
 * edge's tensor that consumer v needs on device d, A(u,d) the part producer u
 * holds there:
 *   forward  = max_d |A(v,d)| - |A(v,d) n A(u,d)|
 *   backward = max_d |A(u,d)| - |A(u,d) n A(v,d)|   (the gradient flows back)
 *   out      = r * (ceil(forward) + ceil(backward))  in words.
 * Device d of a configuration with P = prod s_k devices is the grid point
 * whose mixed-radix digits (loop dim 0 slowest) spell d; devices d >= P take
 * no part.  A tensor dim is cut into s equal parts on each side by the split s
 * of the loop dim it maps to there (1 when unmapped, so loop dims that no
 * tensor dim maps to replicate); a part is then a box of fractions of the
 * tensor.  Fractions are counted exactly on a grid of L_t = s_u * s_v cells
 * per tensor dim (cell c lies in part floor(c * s / L_t) of a side). */
static int transfer_volume(oracle_t *o, int e, const uint32_t *su_, const uint32_t *sv_, uint64_t *out) {
    int u = o->src[e], v = o->dst[e], R = o->rank[e];
    uint64_t Pu = 1, Pv = 1;
    for (int k = 0; k < o->ndims[u]; k++) Pu *= su_[k];
    for (int k = 0; k < o->ndims[v]; k++) Pv *= sv_[k];
    uint64_t su[MAXD], sv[MAXD];
    unsigned __int128 cells = 1;                 /* grid cells of the whole tensor */
    for (int t = 0; t < R; t++) {
        int a = o->src_dim[e * MAXD + t], b = o->dst_dim[e * MAXD + t];
        su[t] = a >= 0 ? su_[a] : 1;
        sv[t] = b >= 0 ? sv_[b] : 1;
        cells *= (unsigned __int128)(su[t] * sv[t]);
    }
    unsigned __int128 fwd = 0, bwd = 0;          /* in cells */
    for (uint64_t d = 0; d < (Pu > Pv ? Pu : Pv); d++) {
        int on_u = d < Pu, on_v = d < Pv;
        uint64_t xu_loop[MAXD] = {0}, xv_loop[MAXD] = {0}, x;
        x = d;
        for (int k = o->ndims[u] - 1; k >= 0; k--) { xu_loop[k] = x % su_[k]; x /= su_[k]; }
        x = d;
        for (int k = o->ndims[v] - 1; k >= 0; k--) { xv_loop[k] = x % sv_[k]; x /= sv_[k]; }
        unsigned __int128 need_v = 1, hold_u = 1, common = 1;
        for (int t = 0; t < R; t++) {
            int a = o->src_dim[e * MAXD + t], b = o->dst_dim[e * MAXD + t];
            uint64_t xu = a >= 0 ? xu_loop[a] : 0, xv = b >= 0 ? xv_loop[b] : 0;
            uint64_t L = su[t] * sv[t], nv_ = 0, nu_ = 0, both = 0;
            for (uint64_t c = 0; c < L; c++) {
                int in_v = c * sv[t] / L == xv, in_u = c * su[t] / L == xu;
                nv_ += in_v;
                nu_ += in_u;
                both += in_v && in_u;
            }
            need_v *= nv_;
            hold_u *= nu_;
            common *= both;
        }
        unsigned __int128 f = on_v ? need_v - (on_u ? common : 0) : 0;
        unsigned __int128 g = on_u ? hold_u - (on_v ? common : 0) : 0;
        if (f > fwd) fwd = f;
        if (g > bwd) bwd = g;
    }
    unsigned __int128 E = o->elems[e];
    unsigned __int128 words = (E * fwd + cells - 1) / cells + (E * bwd + cells - 1) / cells;
    if (words >> 64) return 0;
    return mul_ok(o->r, (uint64_t)words, out);
}

/* Transfer cost model for the next configuration enumeration. */
int oracle_set_transfer_model(oracle_t *o, int model) {
    if (model < 0 || model > 1) return fail(o, "transfer model 0 or 1");
    o->xmodel = model;
    return 0;
}

/* Enumerate C(v) for every v and fill the cost tables. */
static int configs(oracle_t *o, int p, int pow2) {
    free_tables(o);
    free_configs(o);
    o->solved = 0;
    if (p < 1) return fail(o, "p must be positive");
    if (pow2 && (p & (p - 1))) return fail(o, "p must be a power of two");
    o->p = p;
    o->K = calloc(o->nv, sizeof(int));
    o->sp = calloc(o->nv, sizeof(uint32_t *));
    o->Lc = calloc(o->nv, sizeof(uint64_t *));
    o->Rx = calloc(o->ne + 1, sizeof(uint64_t *));
    const int cap = 65535;   /* argmins are uint16 */
    for (int v = 0; v < o->nv; v++) {
        int d = o->ndims[v];
        uint32_t cur[MAXD];
        int count = 0;
        if (!enum_rec(d, 0, (uint64_t)p, pow2, cur, NULL, &count, cap))
            return fail(o, "too many configurations for a uint16 argmin");
        o->sp[v] = calloc((size_t)count * d, sizeof(uint32_t));
        count = 0;
        enum_rec(d, 0, (uint64_t)p, pow2, cur, o->sp[v], &count, cap);
        o->K[v] = count;
        o->Lc[v] = calloc(count, sizeof(uint64_t));
        for (int c = 0; c < count; c++)
            if (!layer_cost(o, v, o->sp[v] + (size_t)c * d, &o->Lc[v][c]))
                return fail(o, "layer cost overflows uint64");
    }
    int bad = 0;
    for (int e = 0; e < o->ne; e++)
        o->Rx[e] = calloc((size_t)o->K[o->src[e]] * o->K[o->dst[e]], sizeof(uint64_t));
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic) reduction(| : bad)
#endif
    for (int e = 0; e < o->ne; e++) {
        int u = o->src[e], v = o->dst[e];
        for (int cu = 0; cu < o->K[u]; cu++)
            for (int cv = 0; cv < o->K[v]; cv++) {
                const uint32_t *a = o->sp[u] + (size_t)cu * o->ndims[u], *b = o->sp[v] + (size_t)cv * o->ndims[v];
                uint64_t *x = &o->Rx[e][(size_t)cu * o->K[v] + cv];
                if (!(o->xmodel ? transfer_volume(o, e, a, b, x) : transfer_cost(o, e, a, b, x))) bad = 1;
            }
    }
    if (bad) return fail(o, "transfer cost overflows uint64");
    return 0;
}

/* Power-of-two splits only, p = 2^L. */
int oracle_configs(oracle_t *o, int p) { return configs(o, p, 1); }

/* Every tuple of positive integers with product <= p (Sec. II's C(v)). */
int oracle_configs_all(oracle_t *o, int p) { return configs(o, p, 0); }

/* Replace the cost tables by caller-given ones (tests with random costs).
 * layer: concatenation of K_v values per vertex; edge: concatenation of the
 * row-major K_src x K_dst matrices per edge. */
int oracle_set_costs(oracle_t *o, const uint64_t *layer, const uint64_t *edge) {
    if (!o->K) return fail(o, "configs not enumerated");
    free_tables(o);
    o->solved = 0;
    size_t off = 0;
    for (int v = 0; v < o->nv; v++)
        for (int c = 0; c < o->K[v]; c++) o->Lc[v][c] = layer[off++];
    off = 0;
    for (int e = 0; e < o->ne; e++) {
        size_t n = (size_t)o->K[o->src[e]] * o->K[o->dst[e]];
        for (size_t k = 0; k < n; k++) o->Rx[e][k] = edge[off++];
    }
    return 0;
}

/* --------------------------------------------------------- ordering */


/* The component of u in the subgraph induced by the vertices marked in `in`
 * (u itself included whatever its mark): comp[] receives 1 for its members.
 * Returns the member count. */
static int component(oracle_t *o, const char *in, int u, char *comp, int *stack) {
    int n = o->nv, top = 0, size = 0;
    memset(comp, 0, n);
    comp[u] = 1;
    stack[top++] = u;
    while (top) {
        int x = stack[--top];
        size++;
        for (int k = 0; k < o->deg[x]; k++) {
            int y = o->nbr[x][k];
            if (in[y] && !comp[y]) { comp[y] = 1; stack[top++] = y; }
        }
    }
    return size;
}

/* The dependent set (Sec. III-B) that u has when it follows the vertices
 * marked in `placed`: the neighbours, neither placed nor u, of u's component
 * in the subgraph induced by placed + {u}.  dep[] receives 1 for its members;
 * returns its size. */
static int dependents_after(oracle_t *o, char *placed, int u, char *dep, char *comp, int *stack) {
    int n = o->nv, size = 0;
    char was = placed[u];
    placed[u] = 1;
    component(o, placed, u, comp, stack);
    placed[u] = was;
    memset(dep, 0, n);
    for (int x = 0; x < n; x++) {
        if (!comp[x]) continue;
        for (int k = 0; k < o->deg[x]; k++) {
            int y = o->nbr[x][k];
            if (!placed[y] && y != u && !dep[y]) { dep[y] = 1; size++; }
        }
    }
    return size;
}

/* GenerateSeq (Fig. 3), a greedy order: each step places the unplaced vertex
 * with the smallest d-set, ties to the lowest vertex id.  The paper keeps the
 * d-sets up to date by merging the chosen vertex's set into its members' sets;
 * by Theorem 2 a vertex's d-set is then exactly the dependent set it would
 * have if placed next, which is what this evaluates.  rule 0: that is the size
 * compared.  rule 1 (the merge as printed, which does not remove a member from
 * its own set): a vertex enters its own d-set when a placed vertex merges into
 * it -- exactly when it has a placed neighbour -- and counts itself from then
 * on.  D(i) is the chosen vertex's dependent set. */
static void generate_seq(oracle_t *o, int rule) {
    int n = o->nv;
    char *placed = calloc(n, 1), *dep = calloc(n, 1), *comp = calloc(n, 1);
    int *stack = calloc(n, sizeof(int));
    for (int i = 0; i < n; i++) {
        int best = -1, best_sz = 0;
        for (int u = 0; u < n; u++) {
            if (placed[u]) continue;
            int sz = dependents_after(o, placed, u, dep, comp, stack);
            if (rule == 1) {
                int placed_neighbour = 0;
                for (int k = 0; k < o->deg[u]; k++) placed_neighbour |= placed[o->nbr[u][k]];
                sz += placed_neighbour;
            }
            if (best < 0 || sz < best_sz) { best = u; best_sz = sz; }
        }
        o->seq[i] = best;
        o->pos[best] = i;
        placed[best] = 1;
    }
    free(placed); free(dep); free(comp); free(stack);
}

/* D(i) for every position of the order in seq[] / pos[], from the definition:
 * the dependent set of v_i after the vertices of positions < i (ascending
 * vertex ids). */
static void dependent_sets(oracle_t *o) {
    int n = o->nv;
    char *placed = calloc(n, 1), *dep = calloc(n, 1), *comp = calloc(n, 1);
    int *stack = calloc(n, sizeof(int));
    for (int i = 0; i < n; i++) {
        dependents_after(o, placed, o->seq[i], dep, comp, stack);
        o->nD[i] = 0;
        for (int v = 0; v < n; v++) if (dep[v]) o->D[i][o->nD[i]++] = v;
        placed[o->seq[i]] = 1;
    }
    free(placed); free(dep); free(comp); free(stack);
}

/* --------------------------------------------------------- dynamic program */

/* Canonical index of phi restricted to D(j), read from a full assignment. */
static uint64_t table_index(oracle_t *o, int j, const int *cfg_of) {
    uint64_t idx = 0;
    for (int k = 0; k < o->nD[j]; k++) idx = idx * (uint64_t)o->K[o->D[j][k]] + (uint64_t)cfg_of[o->D[j][k]];
    return idx;
}

/* Node function H_V(i, phi') of eq. (3): layer cost of v_i plus r*t_x for
 * every edge joining v_i and a vertex later in the sequence (each edge of a
 * multigraph counted, as in the sum over E of eq. 1). */
static int node_cost(oracle_t *o, int i, const int *later_edges, int nlater, const int *cfg_of,
                     uint64_t *out) {
    int vi = o->seq[i];
    uint64_t cost = o->Lc[vi][cfg_of[vi]];
    for (int k = 0; k < nlater; k++) {
        int e = later_edges[k], u = o->src[e], v = o->dst[e];
        uint64_t x = o->Rx[e][(size_t)cfg_of[u] * o->K[v] + cfg_of[v]];
        if (!add_ok(cost, x, &cost)) return 0;
    }
    *out = cost;
    return 1;
}

/* Entries of every table (product of K over D(i)) and the cell count; 0 when
 * a table would exceed 2^34 entries (the oracle keeps every table in memory). */
static int table_sizes(oracle_t *o) {
    o->cells = 0;
    for (int i = 0; i < o->nv; i++) {
        uint64_t N = 1;
        for (int k = 0; k < o->nD[i]; k++)
            if (!mul_ok(N, (uint64_t)o->K[o->D[i][k]], &N) || N > ((uint64_t)1 << 34)) return 0;
        o->N[i] = N;
        o->cells += N * (uint64_t)o->K[o->seq[i]];
    }
    return 1;
}

/* Back-substitution from the last position: c_i = A_i[phi restricted to
 * D(i)], every vertex of D(i) being later in the sequence. */
static void back_substitute(oracle_t *o) {
    int n = o->nv;
    o->min_cost = o->T[n - 1][0];
    int *cfg_of = calloc(n, sizeof(int));
    for (int i = n - 1; i >= 0; i--) {
        uint64_t idx = table_index(o, i, cfg_of);
        cfg_of[o->seq[i]] = o->A[i][idx];
    }
    for (int v = 0; v < n; v++) o->strategy[v] = cfg_of[v];
    free(cfg_of);
    o->solved = 1;
}

/* S(i) of recurrence (4): the components of X(i) - {v_i}, X(i) being v_i's
 * component among the vertices of positions <= i.  Each component is the
 * connected set X(j) of its last position j (Sec. III-B), so its optimum for
 * a given assignment of D(j) is the table R(j, .).  sub[] receives those
 * positions j; returns their count. */
static int subproblems(oracle_t *o, int i, int *sub, char *before, char *X, char *Y, char *taken, int *stack) {
    int n = o->nv, nsub = 0;
    for (int v = 0; v < n; v++) before[v] = o->pos[v] < i;
    component(o, before, o->seq[i], X, stack);   /* X(i) */
    memset(taken, 0, n);
    for (int x = 0; x < n; x++) {
        if (!X[x] || x == o->seq[i] || taken[x]) continue;
        component(o, before, x, Y, stack);       /* one component of X(i) - {v_i} */
        int j = -1;
        for (int y = 0; y < n; y++)
            if (Y[y]) { taken[y] = 1; if (o->pos[y] > j) j = o->pos[y]; }
        sub[nsub++] = j;
    }
    return nsub;
}

/* One entry of recurrence (4): with an assignment phi of D(i) in cfg_of,
 *   R(i, phi) = min over c in C(v_i) of  H(i, phi + {v_i: c})
 *               + sum over j in S(i) of R(j, (phi + {v_i: c}) restricted to D(j)),
 * H being the node function of eq. (3).  Configurations are tried in
 * ascending index order and the first smallest wins.  Returns 0 when a sum
 * overflows uint64. */
static int recurrence_entry(oracle_t *o, int i, const int *sub, int nsub, const int *later, int nlater,
                            int *cfg_of, uint64_t *value, int *arg) {
    int vi = o->seq[i];
    uint64_t best = 0;
    int best_c = 0;
    for (int c = 0; c < o->K[vi]; c++) {
        cfg_of[vi] = c;
        uint64_t cand;
        if (!node_cost(o, i, later, nlater, cfg_of, &cand)) return 0;
        for (int t = 0; t < nsub; t++) {   /* the subproblems' optima */
            int j = sub[t];
            if (!add_ok(cand, o->T[j][table_index(o, j, cfg_of)], &cand)) return 0;
        }
        if (c == 0 || cand < best) { best = cand; best_c = c; }
    }
    *value = best;
    *arg = best_c;
    return 1;
}

/* FindBestStrategy (Fig. 4).  order: NULL -> GenerateSeq with `rule`, else the
 * given sequence of vertex ids (dependent sets then come from their
 * definition).  max_cells > 0 stops after the first vertex that reaches that
 * many cell evaluations (a timing sample; the result is then partial).
 * nthreads > 0 runs the loop over phi on that many OpenMP threads; the loop
 * over configurations stays sequential, so the tie-break is unchanged. */
int oracle_solve(oracle_t *o, int rule, const int *order, uint64_t max_cells, int nthreads) {
    if (!o->K) return fail(o, "configs not enumerated");
    free_tables(o);
    int n = o->nv;
    o->seq = calloc(n, sizeof(int)); o->pos = calloc(n, sizeof(int));
    o->D = calloc(n, sizeof(int *)); o->nD = calloc(n, sizeof(int));
    for (int i = 0; i < n; i++) o->D[i] = calloc(n, sizeof(int));
    o->N = calloc(n, sizeof(uint64_t));
    o->T = calloc(n, sizeof(uint64_t *)); o->A = calloc(n, sizeof(uint16_t *));
    o->strategy = calloc(n, sizeof(int));
    o->solved = 0; o->overflow = 0; o->cells_done = 0;

    char *all = calloc(n, 1), *X = calloc(n, 1), *Y = calloc(n, 1), *taken = calloc(n, 1);
    int *stack = calloc(n, sizeof(int));
    /* weak connectivity (the paper's computation graphs are weakly connected) */
    memset(all, 1, n);
    if (component(o, all, 0, X, stack) != n) {
        free(all); free(X); free(Y); free(taken); free(stack);
        return fail(o, "graph is not weakly connected");
    }

    if (order) {
        char *seen = calloc(n, 1);
        for (int i = 0; i < n; i++) {
            if (order[i] < 0 || order[i] >= n || seen[order[i]]) {
                free(seen); free(all); free(X); free(Y); free(taken); free(stack);
                return fail(o, "bad order");
            }
            seen[order[i]] = 1;
            o->seq[i] = order[i];
            o->pos[order[i]] = i;
        }
        free(seen);
    } else {
        generate_seq(o, rule);
    }
    dependent_sets(o);

    if (!table_sizes(o)) {
        free(all); free(X); free(Y); free(taken); free(stack);
        return fail(o, "table too large");
    }

    int *sub = calloc(n, sizeof(int));
    int *later = calloc(o->ne + 1, sizeof(int));
    struct timespec t0, t1;
    clock_gettime(CLOCK_MONOTONIC, &t0);
    int stopped = 0;

    for (int i = 0; i < n && !stopped; i++) {
        int vi = o->seq[i];
        int nsub = subproblems(o, i, sub, all, X, Y, taken, stack);
        /* the edges H charges to v_i: those joining it to a later vertex */
        int nlater = 0;
        for (int e = 0; e < o->ne; e++) {
            int other = o->src[e] == vi ? o->dst[e] : (o->dst[e] == vi ? o->src[e] : -1);
            if (other >= 0 && o->pos[other] > i) later[nlater++] = e;
        }

        uint64_t N = o->N[i];
        o->T[i] = malloc(N * sizeof(uint64_t));
        o->A[i] = malloc(N * sizeof(uint16_t));
        int nd = o->nD[i];
        const int *Di = o->D[i];
        int ovf = 0;

#ifdef _OPENMP
        int nt = nthreads > 0 ? nthreads : 1;
#pragma omp parallel num_threads(nt) reduction(| : ovf)
#endif
        {
            int *cfg_of = malloc(n * sizeof(int));
            for (int v = 0; v < n; v++) cfg_of[v] = -1;
#ifdef _OPENMP
#pragma omp for schedule(static)
#endif
            for (int64_t phi = 0; phi < (int64_t)N; phi++) {
                /* the assignment of D(i) with canonical index phi (first digit slowest) */
                uint64_t rem = (uint64_t)phi;
                for (int k = nd - 1; k >= 0; k--) {
                    uint64_t Kw = (uint64_t)o->K[Di[k]];
                    cfg_of[Di[k]] = (int)(rem % Kw);
                    rem /= Kw;
                }
                uint64_t value;
                int arg;
                if (!recurrence_entry(o, i, sub, nsub, later, nlater, cfg_of, &value, &arg)) { ovf = 1; continue; }
                o->T[i][phi] = value;
                o->A[i][phi] = (uint16_t)arg;
            }
            free(cfg_of);
        }
        if (ovf) { o->overflow = 1; stopped = 1; break; }
        o->cells_done += N * (uint64_t)o->K[vi];
        if (max_cells && o->cells_done >= max_cells && i + 1 < n) stopped = 2;
    }
    clock_gettime(CLOCK_MONOTONIC, &t1);
    o->seconds = (double)(t1.tv_sec - t0.tv_sec) + 1e-9 * (double)(t1.tv_nsec - t0.tv_nsec);
    free(all); free(X); free(Y); free(taken); free(stack); free(sub); free(later);
    if (o->overflow) return fail(o, "cost overflows uint64");
    if (stopped == 2) return 2;  /* partial run: timing sample only */

    /* R_V(|V|, empty) and back-substitution from the last vertex */
    back_substitute(o);
    return 0;
}

/* The breadth-first recurrence, eq. (2) of Sec. III-A, written as printed:
 * the sequence is a breadth-first traversal from vertex 0 (neighbours taken
 * in ascending id order), D_B(i) = N(V_{<=i}) intersected with V_{>i}, and
 *   B(i, phi) = min over C of  H(i, phi') + B(i-1, phi'|D_B(i-1)),
 *   phi' = phi U {(v_i, C)},  B(before the first position) = 0,
 * with H the node function of eq. (3).  Ties keep the lowest C.  The tables
 * are stored like those of oracle_solve (canonical order over D_B(i)), so the
 * same getters read them; B(|V|, empty) is the minimum and back-substitution
 * recovers the strategy.  max_cells / nthreads as in oracle_solve. */
int oracle_solve_bf(oracle_t *o, uint64_t max_cells, int nthreads) {
    if (!o->K) return fail(o, "configs not enumerated");
    free_tables(o);
    int n = o->nv;
    o->seq = calloc(n, sizeof(int)); o->pos = calloc(n, sizeof(int));
    o->D = calloc(n, sizeof(int *)); o->nD = calloc(n, sizeof(int));
    for (int i = 0; i < n; i++) o->D[i] = calloc(n, sizeof(int));
    o->N = calloc(n, sizeof(uint64_t));
    o->T = calloc(n, sizeof(uint64_t *)); o->A = calloc(n, sizeof(uint16_t *));
    o->strategy = calloc(n, sizeof(int));
    o->solved = 0; o->overflow = 0; o->cells_done = 0;

    /* breadth-first traversal from vertex 0 (nbr[] lists are ascending) */
    char *visited = calloc(n, 1);
    int head = 0, tail = 0;
    o->seq[tail++] = 0;
    visited[0] = 1;
    while (head < tail) {
        int v = o->seq[head++];
        for (int k = 0; k < o->deg[v]; k++) {
            int u = o->nbr[v][k];
            if (!visited[u]) { visited[u] = 1; o->seq[tail++] = u; }
        }
    }
    free(visited);
    if (tail != n) return fail(o, "graph is not weakly connected");
    for (int i = 0; i < n; i++) o->pos[o->seq[i]] = i;

    /* D_B(i) = N(V_{<=i}) intersected with V_{>i}, ascending vertex ids */
    for (int i = 0; i < n; i++) {
        o->nD[i] = 0;
        for (int w = 0; w < n; w++) {
            if (o->pos[w] <= i) continue;
            int adjacent = 0;
            for (int k = 0; k < o->deg[w] && !adjacent; k++) adjacent = o->pos[o->nbr[w][k]] <= i;
            if (adjacent) o->D[i][o->nD[i]++] = w;
        }
    }
    if (!table_sizes(o)) return fail(o, "table too large");

    int *later = calloc(o->ne + 1, sizeof(int));
    struct timespec t0, t1;
    clock_gettime(CLOCK_MONOTONIC, &t0);
    int stopped = 0;
    for (int i = 0; i < n && !stopped; i++) {
        int vi = o->seq[i];
        /* H(i, .) charges the edges joining v_i and a later vertex */
        int nlater = 0;
        for (int e = 0; e < o->ne; e++) {
            int a = o->src[e], b = o->dst[e];
            if ((a == vi && o->pos[b] > i) || (b == vi && o->pos[a] > i)) later[nlater++] = e;
        }
        uint64_t N = o->N[i];
        int Ki = o->K[vi];
        o->T[i] = malloc(N * sizeof(uint64_t));
        o->A[i] = malloc(N * sizeof(uint16_t));
        int nd = o->nD[i];
        const int *Di = o->D[i];
        int ovf = 0;
#ifdef _OPENMP
        int nt = nthreads > 0 ? nthreads : 1;
#pragma omp parallel num_threads(nt) reduction(| : ovf)
#endif
        {
            int *cfg_of = malloc(n * sizeof(int));
            for (int v = 0; v < n; v++) cfg_of[v] = -1;
#ifdef _OPENMP
#pragma omp for schedule(static)
#endif
            for (int64_t phi = 0; phi < (int64_t)N; phi++) {
                uint64_t rem = (uint64_t)phi;
                for (int k = nd - 1; k >= 0; k--) {
                    uint64_t Kw = (uint64_t)o->K[Di[k]];
                    cfg_of[Di[k]] = (int)(rem % Kw);
                    rem /= Kw;
                }
                uint64_t best = UINT64_MAX;
                int arg = 0;
                for (int c = 0; c < Ki; c++) {
                    cfg_of[vi] = c;
                    uint64_t cost;
                    if (!node_cost(o, i, later, nlater, cfg_of, &cost)) { ovf = 1; break; }
                    /* + B(i-1, phi'|D_B(i-1)); D_B(i-1) lies within D_B(i) + {v_i} */
                    if (i > 0 && !add_ok(cost, o->T[i - 1][table_index(o, i - 1, cfg_of)], &cost)) {
                        ovf = 1;
                        break;
                    }
                    if (cost < best) { best = cost; arg = c; }
                }
                o->T[i][phi] = best;
                o->A[i][phi] = (uint16_t)arg;
            }
            free(cfg_of);
        }
        if (ovf) { o->overflow = 1; stopped = 1; break; }
        o->cells_done += N * (uint64_t)Ki;
        if (max_cells && o->cells_done >= max_cells && i + 1 < n) stopped = 2;
    }
    clock_gettime(CLOCK_MONOTONIC, &t1);
    o->seconds = (double)(t1.tv_sec - t0.tv_sec) + 1e-9 * (double)(t1.tv_nsec - t0.tv_nsec);
    free(later);
    if (o->overflow) return fail(o, "cost overflows uint64");
    if (stopped == 2) return 2;
    back_substitute(o);
    return 0;
}

/* --------------------------------------------------------- device assignment */

/* Part g of a configuration with splits s (d loop dims): its grid point, the
 * mixed-radix digits of g with loop dim 0 slowest. */
static void part_digits(const uint32_t *s, int d, uint64_t g, uint64_t *x) {
    for (int k = d - 1; k >= 0; k--) { x[k] = g % s[k]; g /= s[k]; }
}

/* Elements of edge e's tensor that part gu of the source's configuration su
 * and part gw of the destination's configuration sw both cover, rounded down.
 * Per tensor dim the part of a side is the fraction interval [x/s, (x+1)/s)
 * of the loop dim it maps to there (the whole dim when unmapped); the
 * intersection is counted cell by cell on a grid of s_u * s_w cells per dim. */
static uint64_t part_overlap(oracle_t *o, int e, const uint32_t *su, uint64_t gu, const uint32_t *sw, uint64_t gw) {
    int u = o->src[e], w = o->dst[e];
    uint64_t xu[MAXD], xw[MAXD];
    part_digits(su, o->ndims[u], gu, xu);
    part_digits(sw, o->ndims[w], gw, xw);
    unsigned __int128 common = 1, cells = 1;
    for (int t = 0; t < o->rank[e]; t++) {
        int a = o->src_dim[e * MAXD + t], b = o->dst_dim[e * MAXD + t];
        uint64_t au = a >= 0 ? su[a] : 1, aw = b >= 0 ? sw[b] : 1;
        uint64_t pu = a >= 0 ? xu[a] : 0, pw = b >= 0 ? xw[b] : 0;
        uint64_t L = au * aw, both = 0;
        for (uint64_t c = 0; c < L; c++) both += (c * au / L == pu) && (c * aw / L == pw);
        common *= both;
        cells *= L;
    }
    return (uint64_t)(((unsigned __int128)o->elems[e] * common) / cells);
}

/* Elements of edge e's tensor on the source's part gu (side 0) or the
 * destination's part gw (side 1): elems / (product of that side's splits of
 * the mapped dims), counted in the same cells. */
static unsigned __int128 part_cells(oracle_t *o, int e, const uint32_t *su, const uint32_t *sw, int side,
                                    unsigned __int128 *cells) {
    unsigned __int128 mine = 1, all = 1;
    for (int t = 0; t < o->rank[e]; t++) {
        int a = o->src_dim[e * MAXD + t], b = o->dst_dim[e * MAXD + t];
        uint64_t au = a >= 0 ? su[a] : 1, aw = b >= 0 ? sw[b] : 1;
        all *= au * aw;
        mine *= side == 0 ? aw : au;   /* a part of u covers aw of the au * aw cells */
    }
    *cells = all;
    return mine;
}

/* The greedy device assignment of strategy cfg after the search (Sec. II):
 * vertices in ascending id order; the first gets part g on device g; every
 * later one assigns its parts to distinct devices, largest locality first --
 * the locality of (part g, device d) is the elements of the tensors of all
 * edges joining it to an already placed vertex that g and that vertex's part
 * on d both cover -- ties to the lowest part, then the lowest device.
 * dev[v * p + d]: the part of v on device d, -1 for none.  locality[e]: the
 * elements of e's tensor that the two ends hold on the same device, summed
 * over devices.  xfer[e]: r * t_x of e under the assignment, the volume model
 * (forward max_d |need| - |common| plus the same backward, words rounded up
 * per direction) with these devices instead of the grid numbering. */
int oracle_assign_devices(oracle_t *o, const int *cfg, int *dev, uint64_t *locality, uint64_t *xfer) {
    if (!o->K) return fail(o, "configs not enumerated");
    int n = o->nv, p = o->p;
    if (p > 1024) return fail(o, "assignment needs p <= 1024");
    uint64_t *P = calloc(n, sizeof(uint64_t));
    const uint32_t **s = calloc(n, sizeof(uint32_t *));
    for (int v = 0; v < n; v++) {
        if (cfg[v] < 0 || cfg[v] >= o->K[v]) { free(P); free(s); return fail(o, "config out of range"); }
        s[v] = o->sp[v] + (size_t)cfg[v] * o->ndims[v];
        P[v] = 1;
        for (int k = 0; k < o->ndims[v]; k++) P[v] *= s[v][k];
    }
    /* a locality sums the tensors of a vertex's edges: each sum must fit 64 bits */
    uint64_t *esum = calloc(n, sizeof(uint64_t));
    for (int e = 0; e < o->ne; e++)
        if (!add_ok(esum[o->src[e]], o->elems[e], &esum[o->src[e]]) ||
            !add_ok(esum[o->dst[e]], o->elems[e], &esum[o->dst[e]])) {
            free(P); free(s); free(esum);
            return fail(o, "tensor elements of a vertex's edges overflow uint64");
        }
    free(esum);
    for (int i = 0; i < n * p; i++) dev[i] = -1;
    uint64_t *W = calloc((size_t)p * p, sizeof(uint64_t));
    char *gdone = calloc(p, 1), *dused = calloc(p, 1);
    for (int v = 0; v < n; v++) {
        if (v == 0) {
            for (uint64_t g = 0; g < P[v]; g++) dev[v * p + g] = (int)g;
            continue;
        }
        memset(W, 0, (size_t)p * p * sizeof(uint64_t));
        for (int e = 0; e < o->ne; e++) {
            int u = o->src[e], w = o->dst[e];
            int other = u == v ? w : (w == v ? u : -1);
            if (other < 0 || other > v) continue;   /* placed neighbours only */
            for (uint64_t g = 0; g < P[v]; g++)
                for (int d = 0; d < p; d++) {
                    int h = dev[other * p + d];
                    if (h < 0) continue;
                    W[g * p + d] += u == v ? part_overlap(o, e, s[v], g, s[other], (uint64_t)h)
                                           : part_overlap(o, e, s[other], (uint64_t)h, s[v], g);
                }
        }
        memset(gdone, 0, p);
        memset(dused, 0, p);
        for (uint64_t step = 0; step < P[v]; step++) {
            int bg = -1, bd = -1;
            uint64_t best = 0;
            for (uint64_t g = 0; g < P[v]; g++) {
                if (gdone[g]) continue;
                for (int d = 0; d < p; d++) {
                    if (dused[d]) continue;
                    if (bg < 0 || W[g * p + d] > best) { bg = (int)g; bd = d; best = W[g * p + d]; }
                }
            }
            gdone[bg] = 1;
            dused[bd] = 1;
            dev[v * p + bd] = bg;
        }
    }
    for (int e = 0; e < o->ne; e++) {
        int u = o->src[e], w = o->dst[e];
        uint64_t loc = 0;
        unsigned __int128 cells, fwd = 0, bwd = 0;
        unsigned __int128 hold = part_cells(o, e, s[u], s[w], 0, &cells), need = part_cells(o, e, s[u], s[w], 1, &cells);
        for (int d = 0; d < p; d++) {
            int hu = dev[u * p + d], hw = dev[w * p + d];
            unsigned __int128 common_cells = 0;
            if (hu >= 0 && hw >= 0) {
                /* the shared cells of the two parts, counted again exactly */
                uint64_t xu[MAXD], xw[MAXD];
                part_digits(s[u], o->ndims[u], (uint64_t)hu, xu);
                part_digits(s[w], o->ndims[w], (uint64_t)hw, xw);
                common_cells = 1;
                for (int t = 0; t < o->rank[e]; t++) {
                    int a = o->src_dim[e * MAXD + t], b = o->dst_dim[e * MAXD + t];
                    uint64_t au = a >= 0 ? s[u][a] : 1, aw = b >= 0 ? s[w][b] : 1;
                    uint64_t pu = a >= 0 ? xu[a] : 0, pw = b >= 0 ? xw[b] : 0, L = au * aw, both = 0;
                    for (uint64_t c = 0; c < L; c++) both += (c * au / L == pu) && (c * aw / L == pw);
                    common_cells *= both;
                }
                loc += part_overlap(o, e, s[u], (uint64_t)hu, s[w], (uint64_t)hw);
            }
            unsigned __int128 f = hw >= 0 ? need - common_cells : 0, b = hu >= 0 ? hold - common_cells : 0;
            if (f > fwd) fwd = f;
            if (b > bwd) bwd = b;
        }
        locality[e] = loc;
        unsigned __int128 E = o->elems[e];
        unsigned __int128 moved = (E * fwd + cells - 1) / cells + (E * bwd + cells - 1) / cells;
        if (moved >> 64 || !mul_ok(o->r, (uint64_t)moved, &xfer[e])) {
            free(P); free(s); free(W); free(gdone); free(dused);
            return fail(o, "transfer cost overflows uint64");
        }
    }
    free(P); free(s); free(W); free(gdone); free(dused);
    return 0;
}

/* --------------------------------------------------------- getters */

int oracle_num_configs(oracle_t *o, int v) { return o->K ? o->K[v] : -1; }
int oracle_config_splits(oracle_t *o, int v, int c, uint32_t *out) {
    if (!o->K || c < 0 || c >= o->K[v]) return 1;
    memcpy(out, o->sp[v] + (size_t)c * o->ndims[v], o->ndims[v] * sizeof(uint32_t));
    return 0;
}
int oracle_layer_costs(oracle_t *o, int v, uint64_t *out) {
    if (!o->K) return 1;
    memcpy(out, o->Lc[v], o->K[v] * sizeof(uint64_t));
    return 0;
}
int oracle_edge_costs(oracle_t *o, int e, uint64_t *out) {
    if (!o->K) return 1;
    memcpy(out, o->Rx[e], (size_t)o->K[o->src[e]] * o->K[o->dst[e]] * sizeof(uint64_t));
    return 0;
}
int oracle_sequence(oracle_t *o, int *out) {
    if (!o->seq) return 1;
    memcpy(out, o->seq, o->nv * sizeof(int));
    return 0;
}
/* dependent set of the vertex at position i (sorted by vertex id) */
int oracle_dependent_set(oracle_t *o, int i, int *out) {
    if (!o->D) return -1;
    memcpy(out, o->D[i], o->nD[i] * sizeof(int));
    return o->nD[i];
}
uint64_t oracle_table_size(oracle_t *o, int i) { return o->N ? o->N[i] : 0; }
int oracle_table(oracle_t *o, int i, uint64_t *T, uint16_t *A) {
    if (!o->T || !o->T[i]) return 1;
    if (T) memcpy(T, o->T[i], o->N[i] * sizeof(uint64_t));
    if (A) memcpy(A, o->A[i], o->N[i] * sizeof(uint16_t));
    return 0;
}
int oracle_entry(oracle_t *o, int i, uint64_t idx, uint64_t *T, uint32_t *A) {
    if (!o->T || !o->T[i] || idx >= o->N[i]) return 1;
    *T = o->T[i][idx];
    *A = o->A[i][idx];
    return 0;
}
int oracle_result(oracle_t *o, uint64_t *min_cost, int *strategy) {
    if (!o->solved) return 1;
    *min_cost = o->min_cost;
    memcpy(strategy, o->strategy, o->nv * sizeof(int));
    return 0;
}
uint64_t oracle_cells(oracle_t *o) { return o->cells; }
uint64_t oracle_cells_done(oracle_t *o) { return o->cells_done; }
double oracle_seconds(oracle_t *o) { return o->seconds; }
int oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* SplitMix64 output function (Steele, Lea, Flood, OOPSLA 2014). */
static uint64_t splitmix64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

/* Order-independent fingerprints of table i over canonical indices:
 *   fpT = sum_phi mix(mix(phi) ^ T[phi]),  fpA = sum_phi mix(mix(phi) ^ A[phi])
 * (sums mod 2^64). */
int oracle_fingerprint(oracle_t *o, int i, uint64_t *fpT, uint64_t *fpA) {
    if (!o->T || !o->T[i]) return 1;
    uint64_t st = 0, sa = 0;
    for (uint64_t phi = 0; phi < o->N[i]; phi++) {
        uint64_t h = splitmix64_mix(phi);
        st += splitmix64_mix(h ^ o->T[i][phi]);
        sa += splitmix64_mix(h ^ (uint64_t)o->A[i][phi]);
    }
    *fpT = st; *fpA = sa;
    return 0;
}
