"""Seeded synthetic computation graphs for the PaSE strategy search.

This module only *describes* inputs: vertices (a layer's iteration space, which
loop dims are contracted, FLOPs per iteration point) and edges (which tensor
flows, how its dims map onto the loop dims of both endpoints, how many elements
it has).  It contains none of the search method's arithmetic (no configuration
enumeration, no cost model, no ordering, no dynamic program), so both the CPU
oracle and the HIP library can consume it.

Graph dict layout (shared by every consumer)::

    {"name": str, "p": int, "comm_weight": int,
     "vertices": [{"name", "dims": [n_0..n_{d-1}], "dim_names", "reduce": [k..],
                   "flops_per_point": int,
                   "weight_dims": [k..], "weight_per_point": int}],   # optional
     "edges": [{"src", "dst", "src_dim": [..], "dst_dim": [..], "elems": int}]}

``weight_dims`` (optional) name the loop dims that index the layer's weight
tensor, which holds ``weight_per_point`` words per point of those dims (a
k x k convolution: 9 per (co, ci) pair); layers without weights omit both.
``halo`` (optional, convolutions) gives per loop dim the half extent of the
kernel along it (1 for a 3x3 kernel's h and w, 0 elsewhere) and
``input_dims`` the loop dims that index the layer's input tensor
((b, ci, h, w) of a convolution).
``src_dim[k]`` / ``dst_dim[k]`` give, for tensor dim k, the loop dim of the
source / destination vertex that indexes it (-1: that endpoint does not split
this tensor dim).  Vertex ids are list positions; they are the tie-break of the
vertex ordering, so the creation order below is part of each workload.

The five named workloads stand in for the paper's benchmark graphs (AlexNet /
InceptionV3 / RNNLM / Transformer, Sec. IV), whose exact graphs and analytic
cost formulas the paper does not print.  They follow the paper's batch sizes
(128 for CNNs, 64 otherwise) and structure (path graphs, inception modules with
concat fan-in, recurrent grids, encoder-decoder attention with long-lived
encoder output).
"""
from __future__ import annotations

import numpy as np


class _Builder:
    def __init__(self, name: str, p: int, comm_weight: int = 8):
        self.g = {"name": name, "p": int(p), "comm_weight": int(comm_weight),
                  "vertices": [], "edges": []}

    def vertex(self, name, dims, dim_names, reduce, flops_per_point, weights=None, conv=None):
        """weights: (loop dims indexing the weight tensor, words per point);
        conv: (halo width per loop dim, loop dims indexing the input tensor)."""
        assert len(dims) == len(dim_names)
        vx = {"name": name, "dims": [int(x) for x in dims],
              "dim_names": list(dim_names), "reduce": sorted(int(k) for k in reduce),
              "flops_per_point": int(flops_per_point)}
        if weights is not None:
            vx["weight_dims"] = sorted(int(k) for k in weights[0])
            vx["weight_per_point"] = int(weights[1])
        if conv is not None:
            vx["halo"] = [int(w) for w in conv[0]]
            vx["input_dims"] = sorted(int(k) for k in conv[1])
        self.g["vertices"].append(vx)
        return len(self.g["vertices"]) - 1

    def edge(self, src, dst, src_dim, dst_dim, elems=None):
        assert len(src_dim) == len(dst_dim)
        if elems is None:  # size of the tensor produced by src
            sdims = self.g["vertices"][src]["dims"]
            elems = 1
            for k in src_dim:
                if k >= 0:
                    elems *= sdims[k]
        self.g["edges"].append({"src": int(src), "dst": int(dst),
                                "src_dim": [int(k) for k in src_dim],
                                "dst_dim": [int(k) for k in dst_dim],
                                "elems": int(elems)})

    def done(self):
        return self.g


# ---------------------------------------------------------------- W0
def fc_chain(p: int = 4, layers: int = 4, batch: int = 64, width: int = 256):
    """Chain of fully-connected layers (a path graph, like AlexNet's FC tail).

    Loop dims (batch, out, in); the contraction dim is `in`; 2 FLOPs per point.
    The activation (batch, feature) flows from `out` of one layer to `in` of
    the next.
    """
    b = _Builder(f"fc_chain{layers}_b{batch}_w{width}_p{p}", p)
    ids = [b.vertex(f"fc{k}", (batch, width, width), ("b", "out", "in"), (2,), 2, ((1, 2), 1))
           for k in range(layers)]
    for u, v in zip(ids, ids[1:]):
        b.edge(u, v, (0, 1), (0, 2))
    return b.done()


# ---------------------------------------------------------------- W1
_CONV_DIMS = ("b", "co", "ci", "h", "w")


def _conv(k):
    """Halo widths and input dims of a k x k convolution over _CONV_DIMS."""
    return (0, 0, 0, k // 2, k // 2), (0, 2, 3, 4)
_CHANNELS_W1 = (64, 128, 256, 512)


def residual_cnn(seed: int = 0, p: int = 8, layers: int = 16, batch: int = 128):
    """16 3x3 convolutions with a skip edge k -> k+2 for every even k.

    Loop dims (b, co, ci, h, w), contraction over ci, 2*3*3 FLOPs per point.
    Channels are drawn uniformly from {64,128,256,512} (ci of layer 0 first,
    then co of every layer); spatial 64x64 for the first half, 32x32 after.
    """
    rng = np.random.default_rng(seed)
    ci0 = int(rng.choice(_CHANNELS_W1))
    cos = [int(rng.choice(_CHANNELS_W1)) for _ in range(layers)]
    b = _Builder(f"residual_cnn{layers}_seed{seed}_p{p}", p)
    ids = []
    ci = ci0
    for k in range(layers):
        hw = 64 if k < layers // 2 else 32
        ids.append(b.vertex(f"conv{k}", (batch, cos[k], ci, hw, hw), _CONV_DIMS, (2,), 18, ((1, 2), 9),
                            _conv(3)))
        ci = cos[k]
    # activation (b, c, h, w): producer dims (b, co, h, w) -> consumer (b, ci, h, w)
    for k in range(layers - 1):
        b.edge(ids[k], ids[k + 1], (0, 1, 3, 4), (0, 2, 3, 4))
    for k in range(0, layers - 2, 2):
        b.edge(ids[k], ids[k + 2], (0, 1, 3, 4), (0, 2, 3, 4))
    return b.done()


# ---------------------------------------------------------------- W2
_CHANNELS_W2 = (32, 64, 128, 256, 384)


def inception(seed: int = 0, p: int = 16, modules: int = 12, batch: int = 128):
    """Stem conv, `modules` inception modules, final FC.

    Each module has 4 parallel branches of depth U{1,2,3}; every conv has a
    kernel size in U{1,3,5} (2*k*k FLOPs per point) and out-channels in
    U{32,64,128,256,384}.  Branch outputs join in a channel concat vertex with
    loop dims (b, c, h, w) and no contraction.  Spatial size is 35 for the
    first third of the modules, 17 for the second, 8 for the last.
    """
    rng = np.random.default_rng(seed)
    b = _Builder(f"inception{modules}_seed{seed}_p{p}", p)
    stem = b.vertex("stem", (batch, 192, 3, 35, 35), _CONV_DIMS, (2,), 18, ((1, 2), 9), _conv(3))
    x, x_is_concat, cin = stem, False, 192
    third = modules // 3
    for m in range(modules):
        hw = 35 if m < third else (17 if m < 2 * third else 8)
        ends, cout_total = [], 0
        for br in range(4):
            depth = int(rng.integers(1, 4))
            prev, prev_c, prev_is_concat = x, cin, x_is_concat
            for dl in range(depth):
                ksz = int(rng.choice((1, 3, 5)))
                co = int(rng.choice(_CHANNELS_W2))
                v = b.vertex(f"m{m}_b{br}_c{dl}_k{ksz}", (batch, co, prev_c, hw, hw),
                             _CONV_DIMS, (2,), 2 * ksz * ksz, ((1, 2), ksz * ksz), _conv(ksz))
                src = (0, 1, 2, 3) if prev_is_concat else (0, 1, 3, 4)
                b.edge(prev, v, src, (0, 2, 3, 4))
                prev, prev_c, prev_is_concat = v, co, False
            ends.append(prev)
            cout_total += prev_c
        cat = b.vertex(f"m{m}_concat", (batch, cout_total, hw, hw), ("b", "c", "h", "w"), (), 0)
        for e in ends:
            b.edge(e, cat, (0, 1, 3, 4), (0, 1, 2, 3))
        x, x_is_concat, cin = cat, True, cout_total
    fc = b.vertex("fc", (batch, 1000, cin), ("b", "out", "in"), (2,), 2, ((1, 2), 1))
    # pooled features: batch and channels map onto the FC, spatial dims do not
    hw_last = b.g["vertices"][x]["dims"][2]
    b.edge(x, fc, (0, 1, 2, 3), (0, 2, -1, -1), elems=batch * cin * hw_last * hw_last)
    return b.done()


# ---------------------------------------------------------------- W3
def lstm_grid(p: int = 32, layers: int = 2, steps: int = 20, batch: int = 64,
              hidden: int = 2048, vocab: int = 65536):
    """Unrolled multi-layer LSTM language model (a grid DAG) + softmax projection.

    Cell (l, t) is one GEMM with loop dims (b, gate-out = 4*hidden,
    in = input + hidden) contracted over `in`.  Hidden state (b, hidden) flows
    to (l, t+1) and (l+1, t); every top-layer cell feeds the projection GEMM
    (b*steps, vocab, hidden).
    """
    b = _Builder(f"lstm{layers}x{steps}_h{hidden}_p{p}", p)
    cell = {}
    for l in range(layers):
        for t in range(steps):
            cell[l, t] = b.vertex(f"cell_l{l}_t{t}", (batch, 4 * hidden, 2 * hidden),
                                  ("b", "gate", "in"), (2,), 2, ((1, 2), 1))
    hid_elems = batch * hidden
    for l in range(layers):
        for t in range(steps):
            if t + 1 < steps:
                b.edge(cell[l, t], cell[l, t + 1], (0, 1), (0, 2), elems=hid_elems)
            if l + 1 < layers:
                b.edge(cell[l, t], cell[l + 1, t], (0, 1), (0, 2), elems=hid_elems)
    proj = b.vertex("proj", (batch * steps, vocab, hidden), ("bs", "vocab", "in"), (2,), 2, ((1, 2), 1))
    for t in range(steps):
        b.edge(cell[layers - 1, t], proj, (0, 1), (0, 2), elems=hid_elems)
    return b.done()


# ---------------------------------------------------------------- W4
def transformer(p: int = 64, enc_layers: int = 6, dec_layers: int = 6, d_model: int = 1024,
                heads: int = 16, ffn: int = 4096, seq: int = 256, batch: int = 64,
                vocab: int = 32768):
    """Transformer encoder-decoder at the granularity of GEMM-like operators.

    Loop dims use the names b (batch), s (query sequence), h (head), o (out
    feature), i (contracted feature), d (model dim), v (vocabulary).  Per
    encoder layer: fused QKV projection, attention scores, context, output
    projection (contracting heads and head dim), layernorm, FFN up, FFN down,
    layernorm, with residual edges into both layernorms.  Decoder layers add a
    cross-attention block whose key/value projection reads the encoder output.
    """
    b = _Builder(f"transformer{enc_layers}+{dec_layers}_d{d_model}_p{p}", p)
    B, S, H, D, F, V = batch, seq, heads, d_model, ffn, vocab
    dk = D // H
    BSD = ("b", "s", "d")
    ATT = ("b", "s", "h", "o", "i")

    def ln(name):   # residual add + layernorm; gain and bias per model dim
        return b.vertex(name, (B, S, D), BSD, (), 8, ((2,), 2))

    def self_attention(x, pre):
        qkv = b.vertex(pre + "qkv", (B, S, H, 3 * dk, D), ATT, (4,), 2, ((2, 3, 4), 1))
        score = b.vertex(pre + "score", (B, S, H, S, dk), ATT, (4,), 2)
        ctx = b.vertex(pre + "ctx", (B, S, H, dk, S), ATT, (4,), 2)
        oproj = b.vertex(pre + "oproj", (B, S, H, D, dk), ATT, (2, 4), 2, ((2, 3, 4), 1))
        ln1 = ln(pre + "ln1")
        b.edge(x, qkv, (0, 1, 2), (0, 1, 4))           # (b,s,d) -> qkv (b,s,i)
        b.edge(qkv, score, (0, 1, 2, 3), (0, 1, 2, 4))  # Q (b,s,h,dk) -> score (b,s,h,i)
        b.edge(qkv, ctx, (0, 1, 2, 3), (0, 4, 2, 3))    # V (b,s_k,h,dk) -> ctx (b,i,h,o)
        b.edge(score, ctx, (0, 1, 2, 3), (0, 1, 2, 4))  # P (b,s,h,s_k) -> ctx (b,s,h,i)
        b.edge(ctx, oproj, (0, 1, 2, 3), (0, 1, 2, 4))  # (b,s,h,dv) -> oproj (b,s,h,i)
        b.edge(oproj, ln1, (0, 1, 3), (0, 1, 2))        # (b,s,d)
        b.edge(x, ln1, (0, 1, 2), (0, 1, 2))            # residual
        return ln1

    def ffn_block(x, pre, out_name):
        f1 = b.vertex(pre + "ffn1", (B, S, F, D), ("b", "s", "o", "i"), (3,), 2, ((2, 3), 1))
        f2 = b.vertex(pre + "ffn2", (B, S, D, F), ("b", "s", "o", "i"), (3,), 2, ((2, 3), 1))
        out = ln(pre + out_name)
        b.edge(x, f1, (0, 1, 2), (0, 1, 3))
        b.edge(f1, f2, (0, 1, 2), (0, 1, 3))
        b.edge(f2, out, (0, 1, 2), (0, 1, 2))
        b.edge(x, out, (0, 1, 2), (0, 1, 2))            # residual
        return out

    src = b.vertex("src_emb", (B, S, D, V), ("b", "s", "d", "v"), (3,), 2, ((2, 3), 1))
    x = src
    for l in range(enc_layers):
        pre = f"enc{l}_"
        x = ffn_block(self_attention(x, pre), pre, "ln2")
    enc_out = x

    y = b.vertex("tgt_emb", (B, S, D, V), ("b", "s", "d", "v"), (3,), 2, ((2, 3), 1))
    for l in range(dec_layers):
        pre = f"dec{l}_"
        ln1 = self_attention(y, pre)
        xq = b.vertex(pre + "xq", (B, S, H, dk, D), ATT, (4,), 2, ((2, 3, 4), 1))
        xkv = b.vertex(pre + "xkv", (B, S, H, 2 * dk, D), ATT, (4,), 2, ((2, 3, 4), 1))
        xscore = b.vertex(pre + "xscore", (B, S, H, S, dk), ATT, (4,), 2)
        xctx = b.vertex(pre + "xctx", (B, S, H, dk, S), ATT, (4,), 2)
        xoproj = b.vertex(pre + "xoproj", (B, S, H, D, dk), ATT, (2, 4), 2, ((2, 3, 4), 1))
        ln2 = ln(pre + "ln2")
        b.edge(ln1, xq, (0, 1, 2), (0, 1, 4))
        b.edge(enc_out, xkv, (0, 1, 2), (0, 1, 4))
        b.edge(xq, xscore, (0, 1, 2, 3), (0, 1, 2, 4))   # Q
        b.edge(xkv, xscore, (0, 1, 2, 3), (0, 3, 2, 4))  # K (b,s_k,h,dk) -> (b,o,h,i)
        b.edge(xscore, xctx, (0, 1, 2, 3), (0, 1, 2, 4))
        b.edge(xkv, xctx, (0, 1, 2, 3), (0, 4, 2, 3))    # V (b,s_k,h,dk) -> (b,i,h,o)
        b.edge(xctx, xoproj, (0, 1, 2, 3), (0, 1, 2, 4))
        b.edge(xoproj, ln2, (0, 1, 3), (0, 1, 2))
        b.edge(ln1, ln2, (0, 1, 2), (0, 1, 2))           # residual
        y = ffn_block(ln2, pre, "ln3")

    proj = b.vertex("proj", (B, S, V, D), ("b", "s", "v", "d"), (3,), 2, ((2, 3), 1))
    soft = b.vertex("softmax", (B, S, V), ("b", "s", "v"), (), 5)
    b.edge(y, proj, (0, 1, 2), (0, 1, 3))
    b.edge(proj, soft, (0, 1, 2), (0, 1, 2))
    return b.done()


# ---------------------------------------------------------------- named set
WORKLOADS = {
    "w0_fc_chain": lambda seed=0: fc_chain(),
    "w1_residual_cnn": lambda seed=0: residual_cnn(seed),
    "w2_inception": lambda seed=0: inception(seed),
    "w3_lstm_grid": lambda seed=0: lstm_grid(),
    "w4_transformer": lambda seed=0: transformer(),
}


def workload(name: str, seed: int = 0):
    return WORKLOADS[name](seed)


# ---------------------------------------------------------------- small random inputs
def random_graph(seed: int, n: int, p: int = 4, max_dims: int = 3, extra_edges: int = 2,
                 max_size: int = 64, multi_edges: bool = True):
    """Random weakly connected graph with n vertices (a random spanning tree plus
    `extra_edges` further edges, possibly parallel), random loop-dim sizes
    (not necessarily powers of 2), random contraction dims and random tensor
    maps (including unsplit tensor dims)."""
    rng = np.random.default_rng(seed)
    b = _Builder(f"random_n{n}_seed{seed}_p{p}", p)
    for v in range(n):
        d = int(rng.integers(1, max_dims + 1))
        dims = [int(rng.integers(1, max_size + 1)) for _ in range(d)]
        red = [k for k in range(d) if rng.random() < 0.35]
        b.vertex(f"v{v}", dims, [f"x{k}" for k in range(d)], red, int(rng.integers(1, 5)))

    def rand_edge(u, v):
        du = len(b.g["vertices"][u]["dims"])
        dv = len(b.g["vertices"][v]["dims"])
        rank = int(rng.integers(1, max(du, dv) + 1))
        sd = [int(rng.integers(-1, du)) for _ in range(rank)]
        dd = [int(rng.integers(-1, dv)) for _ in range(rank)]
        b.edge(u, v, sd, dd, elems=int(rng.integers(1, 5000)))

    order = rng.permutation(n)
    for k in range(1, n):
        u, v = int(order[k]), int(order[rng.integers(0, k)])
        if rng.random() < 0.5:
            u, v = v, u
        rand_edge(u, v)
    added = 0
    while added < extra_edges and n > 1:
        u, v = (int(x) for x in rng.integers(0, n, size=2))
        if u == v:
            continue
        if not multi_edges and any({e["src"], e["dst"]} == {u, v} for e in b.g["edges"]):
            continue
        rand_edge(u, v)
        added += 1
    _random_weights(b, seed)
    _random_halos(b, seed)
    return b.done()


def _random_weights(b, seed):
    """Give about two thirds of the vertices a weight tensor over a random
    non-empty subset of their loop dims (1..4 words per point).  Drawn from a
    stream of its own, so the rest of the graph does not depend on it."""
    rng = np.random.default_rng([seed, 0x3E1])
    for vx in b.g["vertices"]:
        d = len(vx["dims"])
        if rng.random() < 0.67:
            dims = [k for k in range(d) if rng.random() < 0.6] or [int(rng.integers(0, d))]
            vx["weight_dims"] = dims
            vx["weight_per_point"] = int(rng.integers(1, 5))


def _random_halos(b, seed):
    """Give about half of the vertices a convolution geometry: a random
    non-empty set of input dims, and on some of them a halo width in 1..2.
    Drawn from a stream of its own, so the rest of the graph does not depend
    on it."""
    rng = np.random.default_rng([seed, 0x4A1])
    for vx in b.g["vertices"]:
        d = len(vx["dims"])
        if rng.random() < 0.5:
            ins = [k for k in range(d) if rng.random() < 0.7] or [int(rng.integers(0, d))]
            halo = [int(rng.integers(1, 3)) if (k in ins and rng.random() < 0.5) else 0 for k in range(d)]
            vx["halo"] = halo
            vx["input_dims"] = ins


def random_costs(seed: int, layer_sizes, edge_shapes, hi: int = 4):
    """Seeded small-integer cost arrays in [0, hi): one vector per vertex
    (length given in `layer_sizes`) and one row-major matrix per edge (shape
    given in `edge_shapes`).  Small `hi` makes ties dense, which exercises the
    lowest-index tie-break."""
    rng = np.random.default_rng(seed)
    layer = [rng.integers(0, hi, size=int(k), dtype=np.uint64) for k in layer_sizes]
    edge = [rng.integers(0, hi, size=(int(a), int(c)), dtype=np.uint64) for a, c in edge_shapes]
    return layer, edge


def chain_graph(seed: int, n: int, p: int = 4, max_dims: int = 3, max_size: int = 64):
    """Random path graph v0 - v1 - ... - v_{n-1} (edge directions random)."""
    rng = np.random.default_rng(seed)
    b = _Builder(f"chain_n{n}_seed{seed}_p{p}", p)
    for v in range(n):
        d = int(rng.integers(1, max_dims + 1))
        dims = [int(rng.integers(1, max_size + 1)) for _ in range(d)]
        red = [k for k in range(d) if rng.random() < 0.35]
        b.vertex(f"v{v}", dims, [f"x{k}" for k in range(d)], red, int(rng.integers(1, 5)))
    for v in range(n - 1):
        u, w = (v, v + 1) if rng.random() < 0.5 else (v + 1, v)
        du = len(b.g["vertices"][u]["dims"])
        dw = len(b.g["vertices"][w]["dims"])
        rank = int(rng.integers(1, max(du, dw) + 1))
        b.edge(u, w, [int(rng.integers(-1, du)) for _ in range(rank)],
               [int(rng.integers(-1, dw)) for _ in range(rank)], elems=int(rng.integers(1, 5000)))
    _random_weights(b, seed)
    _random_halos(b, seed)
    return b.done()
