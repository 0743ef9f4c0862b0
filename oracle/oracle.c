/*
 * ORACLE -- test infrastructure only.
 *
 * A plain, slow, destination-centric CPU reference for layer-wise GNN
 * inference (Taurus, arXiv 2607.17374).  Only the test-suite, the smoke
 * check and the benchmark's CPU-baseline leg may load this file; the GPU
 * library never does, and the two share no code.  Everything here is written
 * to be checked by eye against the paper:
 *
 *   - graph storage: CSR by source (Sec. 3.2, "Data Layout"), built by
 *     sorting the (u, v) pairs, plus in-neighbour lists for the gather;
 *   - one layer = Aggregate over in-neighbours then Update and activation
 *     (Sec. 2.1, Eqs. (1)-(2)), evaluated per destination in fp64
 *     with in-neighbours visited in ascending source ID.  The paper states
 *     that source-centric broadcast is semantically equal to this gather for
 *     the same message set, Aggregate and Update (Sec. 3.1), so the gather is
 *     the plain definition of what the GPU path must reach;
 *   - GraphSAGE with mean aggregation and the concatenated update
 *     W [h_agg || h_v] (Sec. 3.9, "SAGEConv");
 *   - GCN with the symmetric normalisation of Kipf and Welling, one self
 *     loop per vertex (the paper cites the model in Sec. 4.1 without
 *     writing its formula; the directed-graph reading is documented below);
 *   - fanout sampling: up to k incoming edges kept per vertex, per layer
 *     (Sec. 3.9, "Sampling-based Inference"), ranked by a counter-based
 *     hash;
 *   - GIN (GINConv, sum aggregation, with a linear or a two-layer
 *     perceptron apply function) and single-head GATConv (Sec. 3.9,
 *     "GATConv"; Sec. 4.1 evaluates both);
 *     sampled GCN layers take the sampled graph's degrees;
 *   - the degree/BFS vertex ordering used as a topology-aware bootstrap
 *     (Sec. 3.8 discusses bandwidth-style bootstraps; the exact ordering
 *     rule is a reading of the text and is stated at or_reorder_bfs), the
 *     RCMK bootstrap and the topology-aware reordering of Alg. 1 (positions
 *     initialised once from the bootstrap and carried across updates), with
 *     the total span C(pi), the dispersion J and the chunk-level residency
 *     profile A(t) (Sec. 3.8);
 *   - a slot-level simulation of a budgeted layer's residency with the
 *     fewest-pending eviction policy (Sec. 3.5.3) and the random, FIFO and
 *     LRU policies it is compared with (Sec. 4).
 *
 * Parity status: every function here is pinned by CPU tests (dense
 * adjacency-matrix products, closed forms, hand-worked small graphs -- Alg. 1
 * worked by hand over two updates among them --, brute force and the
 * published SplitMix64 outputs); none is unpinned.  The fixture generators
 * live outside the oracle and have no external generator to match.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

/* number of OpenMP threads the oracle's parallel loops use */
int or_threads(void) { return omp_get_max_threads(); }

/* ------------------------------------------------------------ helpers ---- */

typedef struct { int32_t a, b; } or_pair;

static int or_pair_cmp(const void* x, const void* y) {
    const or_pair* p = (const or_pair*)x; const or_pair* q = (const or_pair*)y;
    if (p->a != q->a) return p->a < q->a ? -1 : 1;
    if (p->b != q->b) return p->b < q->b ? -1 : 1;
    return 0;
}

/*
 * CSR by source.  Sort the pairs by (u, v); row u then lists the
 * destinations of u's out-edges in ascending order.  Returns 0, or -1 if the
 * list holds a self loop or a repeated pair (the graph must be simple), or
 * -2 on an ID out of range.
 */
int or_build_csr(int64_t n, int64_t e, const int32_t* src, const int32_t* dst,
                 int64_t* row_off, int32_t* col_dst) {
    or_pair* p = (or_pair*)malloc((size_t)(e > 0 ? e : 1) * sizeof(or_pair));
    if (!p) return -3;
    for (int64_t i = 0; i < e; i++) {
        if (src[i] < 0 || src[i] >= n || dst[i] < 0 || dst[i] >= n) { free(p); return -2; }
        p[i].a = src[i]; p[i].b = dst[i];
    }
    qsort(p, (size_t)e, sizeof(or_pair), or_pair_cmp);
    int rc = 0;
    for (int64_t i = 0; i <= n; i++) row_off[i] = 0;
    for (int64_t i = 0; i < e; i++) {
        if (p[i].a == p[i].b) rc = -1;
        if (i > 0 && p[i].a == p[i - 1].a && p[i].b == p[i - 1].b) rc = -1;
        row_off[p[i].a + 1]++;
        col_dst[i] = p[i].b;
    }
    for (int64_t u = 0; u < n; u++) row_off[u + 1] += row_off[u];
    free(p);
    return rc;
}

/*
 * In-neighbour lists: for every destination v, the sources u of its
 * in-edges (u, v) in ascending order, with in_pos[k] = the CSR position of
 * that edge (so per-edge flags can be mapped between the two orders).
 */
int or_build_in_lists(int64_t n, const int64_t* row_off, const int32_t* col_dst,
                      int64_t* in_off, int32_t* in_src, int64_t* in_pos) {
    int64_t e = row_off[n];
    for (int64_t v = 0; v <= n; v++) in_off[v] = 0;
    for (int64_t i = 0; i < e; i++) in_off[col_dst[i] + 1]++;
    for (int64_t v = 0; v < n; v++) in_off[v + 1] += in_off[v];
    int64_t* fill = (int64_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    if (!fill) return -3;
    for (int64_t v = 0; v < n; v++) fill[v] = in_off[v];
    /* walking CSR rows in ascending u appends sources in ascending order */
    for (int64_t u = 0; u < n; u++)
        for (int64_t i = row_off[u]; i < row_off[u + 1]; i++) {
            int64_t k = fill[col_dst[i]]++;
            in_src[k] = (int32_t)u;
            if (in_pos) in_pos[k] = i;
        }
    free(fill);
    return 0;
}

/*
 * In-neighbour lists straight from the edge list, for graphs too large for
 * the sort above: N^-(v) = {u : (u, v) in E}, sources ascending, by counting
 * in-degrees, placing each source, then sorting each list.  Also the
 * out-degree of every vertex.  The pairs are assumed valid and distinct (the
 * generator's promise; the CSR checks below test the GPU's CSR against the
 * same list).  Returns 0, or -3 when out of memory.
 */
static int or_i32_cmp(const void* x, const void* y) {
    int32_t a = *(const int32_t*)x, b = *(const int32_t*)y;
    return (a > b) - (a < b);
}
int or_in_lists_from_edges(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* in_off,
                           int32_t* in_src, int32_t* deg_out) {
    int64_t* fill = (int64_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int64_t));
    if (!fill) return -3;
#pragma omp parallel for schedule(static)
    for (int64_t v = 0; v <= n; v++) in_off[v] = 0;
#pragma omp parallel for schedule(static)
    for (int64_t v = 0; v < n; v++) deg_out[v] = 0;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < e; i++) {
        __atomic_fetch_add(&in_off[dst[i] + 1], 1, __ATOMIC_RELAXED);
        __atomic_fetch_add(&deg_out[src[i]], 1, __ATOMIC_RELAXED);
    }
    for (int64_t v = 0; v < n; v++) in_off[v + 1] += in_off[v];
#pragma omp parallel for schedule(static)
    for (int64_t v = 0; v < n; v++) fill[v] = in_off[v];
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < e; i++) {
        int64_t k = __atomic_fetch_add(&fill[dst[i]], 1, __ATOMIC_RELAXED);
        in_src[k] = src[i];
    }
    free(fill);
#pragma omp parallel for schedule(dynamic, 4096)
    for (int64_t v = 0; v < n; v++) {
        int64_t d = in_off[v + 1] - in_off[v];
        if (d > 1) qsort(in_src + in_off[v], (size_t)d, sizeof(int32_t), or_i32_cmp);
    }
    return 0;
}

/*
 * Order-independent digests of an edge set, for comparing graphs whose
 * arrays are too large to compare or sort on the host: with
 * f(u, v) = mix64(u * 2^32 + v + G) (a bijection of the pair), out[0] = the
 * number of edges, out[1] = the sum and out[2] = the xor of f over the set.
 * Equal sets give equal digests; unequal ones collide with probability about
 * 2^-64.  Over the raw edge list; over a CSR (the edges whose mask bit is set
 * when mask_words is given); over in-neighbour lists (the entries with
 * keep_in set when given).
 */
static uint64_t or_mix64(uint64_t z);
static uint64_t or_pair_digest(uint64_t u, uint64_t v) { return or_mix64((u << 32) + v + 0x9e3779b97f4a7c15ULL); }

void or_digest_edges(int64_t e, const int32_t* src, const int32_t* dst, uint64_t* out) {
    uint64_t sum = 0, x = 0;
#pragma omp parallel for reduction(+ : sum) reduction(^ : x) schedule(static)
    for (int64_t i = 0; i < e; i++) {
        uint64_t h = or_pair_digest((uint64_t)src[i], (uint64_t)dst[i]);
        sum += h;
        x ^= h;
    }
    out[0] = (uint64_t)e; out[1] = sum; out[2] = x;
}

void or_digest_csr(int64_t n, const int64_t* row_off, const int32_t* col_dst, const uint64_t* mask_words,
                   uint64_t* out) {
    uint64_t sum = 0, x = 0, cnt = 0;
#pragma omp parallel for reduction(+ : sum, cnt) reduction(^ : x) schedule(dynamic, 4096)
    for (int64_t u = 0; u < n; u++)
        for (int64_t i = row_off[u]; i < row_off[u + 1]; i++) {
            if (mask_words && !((mask_words[i >> 6] >> (i & 63)) & 1ULL)) continue;
            uint64_t h = or_pair_digest((uint64_t)u, (uint64_t)col_dst[i]);
            sum += h; x ^= h; cnt++;
        }
    out[0] = cnt; out[1] = sum; out[2] = x;
}

void or_digest_in_lists(int64_t n, const int64_t* in_off, const int32_t* in_src, const uint8_t* keep_in,
                        uint64_t* out) {
    uint64_t sum = 0, x = 0, cnt = 0;
#pragma omp parallel for reduction(+ : sum, cnt) reduction(^ : x) schedule(dynamic, 4096)
    for (int64_t v = 0; v < n; v++)
        for (int64_t j = in_off[v]; j < in_off[v + 1]; j++) {
            if (keep_in && !keep_in[j]) continue;
            uint64_t h = or_pair_digest((uint64_t)in_src[j], (uint64_t)v);
            sum += h; x ^= h; cnt++;
        }
    out[0] = cnt; out[1] = sum; out[2] = x;
}

/*
 * Canonical CSR shape: row_off[0] = 0, non-decreasing, row_off[n] = e;
 * every row strictly ascending, in [0, n), no self loop.  Returns 0 or the
 * first violated rule (1 offsets, 2 range, 3 order or repeat, 4 self loop).
 * With the digest equal to the edge list's, such a CSR is the canonical one.
 */
int or_csr_check(int64_t n, int64_t e, const int64_t* row_off, const int32_t* col_dst) {
    if (row_off[0] != 0 || row_off[n] != e) return 1;
    int bad = 0;
#pragma omp parallel for reduction(max : bad) schedule(dynamic, 4096)
    for (int64_t u = 0; u < n; u++) {
        if (row_off[u + 1] < row_off[u]) { bad = bad > 1 ? bad : 1; continue; }
        for (int64_t i = row_off[u]; i < row_off[u + 1]; i++) {
            int32_t v = col_dst[i];
            int r = 0;
            if (v < 0 || v >= n) r = 2;
            else if (i > row_off[u] && col_dst[i - 1] >= v) r = 3;
            else if (v == u) r = 4;
            if (r > bad) bad = r;
        }
    }
    return bad;
}

/* --------------------------------------------------- counter-based hash -- */
/*
 * H(s, t, x1..xk): h = s; for x in (t, x1..xk): h = mix64(h + G + x), with
 * mix64 the SplitMix64 finaliser and G its golden-ratio increment (Steele,
 * Lea and Flood, OOPSLA 2014).  The fanout sampler draws with tag 4.
 */
static uint64_t or_mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}
uint64_t or_hash(uint64_t seed, uint64_t tag, int nargs, const uint64_t* args) {
    uint64_t h = or_mix64(seed + 0x9e3779b97f4a7c15ULL + tag);
    for (int i = 0; i < nargs; i++) h = or_mix64(h + 0x9e3779b97f4a7c15ULL + args[i]);
    return h;
}

/* ------------------------------------------------------ fanout sampler -- */
typedef struct { uint64_t key; int32_t u; int64_t pos; } or_cand;

static int or_cand_cmp(const void* x, const void* y) {
    const or_cand* p = (const or_cand*)x; const or_cand* q = (const or_cand*)y;
    if (p->key != q->key) return p->key < q->key ? -1 : 1;
    return (p->u > q->u) - (p->u < q->u);
}

/*
 * Per-layer fanout mask (Sec. 3.9, "Sampling-based Inference": for fanout k
 * keep up to k incoming edges per vertex and suppress the rest).  In-edge
 * (u, v) of layer `layer` gets the rank key (H(seed, 4, layer, v, u), u); for
 * every v the min(d_in(v), k) smallest keys are kept.  Outputs:
 *   mask_words  ceil(e/64) words, bit i of the CSR edge order set if kept;
 *   keep_in     per in-list entry, 1 if kept (may be NULL);
 *   m_out       |M_layer(v)|, the kept in-degree.
 * k <= 0 keeps everything (exact inference).
 */
void or_sample(int64_t n, const int64_t* row_off, const int64_t* in_off, const int32_t* in_src,
               const int64_t* in_pos, uint64_t seed, int64_t layer, int64_t k,
               uint64_t* mask_words, uint8_t* keep_in, int32_t* m_out) {
    /* mask_words NULL: only keep_in and m_out (row_off and in_pos unused) */
    if (mask_words) memset(mask_words, 0, (size_t)((row_off[n] + 63) / 64) * sizeof(uint64_t));
#pragma omp parallel
    {
        or_cand* buf = NULL;
        int64_t cap = 0;
#pragma omp for schedule(dynamic, 1024)
        for (int64_t v = 0; v < n; v++) {
            int64_t d = in_off[v + 1] - in_off[v];
            int64_t keep = (k <= 0 || d <= k) ? d : k;
            m_out[v] = (int32_t)keep;
            if (d > cap) { cap = d; buf = (or_cand*)realloc(buf, (size_t)cap * sizeof(or_cand)); }
            for (int64_t j = 0; j < d; j++) {
                int32_t u = in_src[in_off[v] + j];
                uint64_t args[3] = {(uint64_t)layer, (uint64_t)v, (uint64_t)u};
                buf[j].key = or_hash(seed, 4, 3, args);
                buf[j].u = u;
                buf[j].pos = in_off[v] + j;
            }
            if (keep < d) qsort(buf, (size_t)d, sizeof(or_cand), or_cand_cmp);
            for (int64_t j = 0; j < d; j++) {
                int kept = j < keep;
                int64_t idx = buf[j].pos;            /* in-list index */
                if (keep_in) keep_in[idx] = (uint8_t)kept;
                if (kept && mask_words) {
                    int64_t p = in_pos[idx];         /* CSR position */
                    __atomic_fetch_or(&mask_words[p >> 6], 1ULL << (p & 63), __ATOMIC_RELAXED);
                }
            }
        }
        free(buf);
    }
}

/* -------------------------------------------------- precision handling -- */
/* storage dtypes: 0 fp32, 1 bf16, 2 fp16 (16-bit ones as raw bit patterns) */
static double or_load(const void* H, int dtype, int64_t idx) {
    if (dtype == 0) return (double)((const float*)H)[idx];
    uint16_t b = ((const uint16_t*)H)[idx];
    if (dtype == 1) {
        uint32_t x = (uint32_t)b << 16; float f; memcpy(&f, &x, 4); return (double)f;
    }
    /* fp16: sign, 5-bit exponent (bias 15), 10-bit fraction */
    int s = b >> 15, ex = (b >> 10) & 31, fr = b & 1023;
    double mag;
    if (ex == 0) mag = ldexp((double)fr, -24);
    else if (ex == 31) mag = fr ? NAN : INFINITY;
    else mag = ldexp((double)(1024 + fr), ex - 25);
    return s ? -mag : mag;
}

/*
 * fp64 -> fp32 (round to nearest even, the C conversion) -> optionally the
 * 16-bit storage type, also round to nearest even.  Written from the IEEE 754
 * definitions: bf16 keeps the top 16 bits of the fp32 pattern; fp16 keeps 10
 * fraction bits with exponent bias 15.
 */
static uint16_t or_to_bf16(float f) {
    uint32_t x; memcpy(&x, &f, 4);
    if ((x & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((x >> 16) | 0x40u);
    uint32_t lower = x & 0xffffu, upper = x >> 16;
    if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u))) upper++;
    return (uint16_t)upper;
}
static uint16_t or_to_f16(float f) {
    double a = fabs((double)f);
    uint16_t sign = signbit(f) ? 0x8000 : 0;
    if (isnan(f)) return 0x7e00;
    if (a >= 65520.0) return sign | 0x7c00;                /* rounds past the largest finite */
    if (a < ldexp(1.0, -14)) {                              /* subnormal: units of 2^-24 */
        double q = a * ldexp(1.0, 24);
        double r = nearbyint(q);                            /* ties to even */
        return sign | (uint16_t)r;
    }
    int ex; double m = frexp(a, &ex);                       /* a = m * 2^ex, m in [0.5, 1) */
    double q = ldexp(m, 11);                                /* 11 significant bits in [1024, 2048) */
    double r = nearbyint(q);
    if (r >= 2048.0) { r = 1024.0; ex += 1; }
    int bexp = ex - 1 + 15;                                 /* value = (r/1024) * 2^(ex-1) */
    return sign | (uint16_t)(bexp << 10) | (uint16_t)((int)r - 1024);
}
void or_round_store(int64_t count, const double* in, int dtype, void* out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; i++) {
        float f = (float)in[i];
        if (dtype == 0) ((float*)out)[i] = f;
        else if (dtype == 1) ((uint16_t*)out)[i] = or_to_bf16(f);
        else ((uint16_t*)out)[i] = or_to_f16(f);
    }
}
void or_widen(int64_t count, const void* in, int dtype, double* out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; i++) out[i] = or_load(in, dtype, i);
}

/* ------------------------------------------------------------- layers ---- */
/*
 * One GNN layer for the destinations listed in dst_ids (all if NULL), in
 * fp64.  H is the layer input (n rows of width d_in, storage dtype h_dtype);
 * W has the paper's orientation (rows = d_out, it maps an input vector to an
 * output vector) and is given in fp64; bias may be NULL.  keep_in selects the
 * propagated in-edges (NULL = all, exact inference).
 *
 * agg 0, GraphSAGE-mean (Sec. 3.9): with M(v) the propagated in-neighbours,
 *     a    = (1/|M(v)|) * sum_{u in M(v)} h_u   (0 when M(v) is empty),
 *     z    = W [a || h_v] + b,  W = [W_agg  W_self],  cols = 2 d_in.
 * agg 1, GCN, symmetric normalisation with one self loop per vertex on the
 *     directed graph: d^_out(u) = d_out(u) + 1, d^_in(v) = d_in(v) + 1,
 *     a    = sum_{u in N-(v)} h_u / sqrt(d^_out(u) d^_in(v))
 *            + h_v / sqrt(d^_out(v) d^_in(v)),
 *     z    = W a + b,  cols = d_in.  deg_out is the out-degree of the graph
 *     the layer propagates over: the full one for exact inference; for a
 *     sampled layer (keep_in) the kept out-degree, and d_in(v) = |M(v)|, so
 *     the normalisation is that of the sampled graph with its self loops.
 * agg 2, GIN (GINConv with a linear apply function and eps = 0, sum
 *     aggregation):
 *     a    = h_v + sum_{u in M(v)} h_u,
 *     z    = W a + b,  cols = d_in.
 * Output: out[i][j] = ReLU(z_j) if relu else z_j, for v = dst_ids[i].
 */
int or_layer(int agg, int64_t n, const int64_t* in_off, const int32_t* in_src,
             const uint8_t* keep_in, const int32_t* deg_out,
             const void* H, int h_dtype, int64_t d_in,
             const double* W, const double* bias, int64_t d_out, int relu,
             int64_t n_dst, const int64_t* dst_ids, double* out) {
    int64_t cols = agg == 0 ? 2 * d_in : d_in;
    int64_t count = dst_ids ? n_dst : n;
    int bad = 0;
#pragma omp parallel
    {
        double* a = (double*)malloc((size_t)cols * sizeof(double));
        if (!a) bad = 1;
#pragma omp for schedule(dynamic, 256)
        for (int64_t i = 0; i < count; i++) {
            if (!a) continue;
            int64_t v = dst_ids ? dst_ids[i] : i;
            for (int64_t j = 0; j < cols; j++) a[j] = 0.0;
            if (agg == 0) {
                int64_t m = 0;
                for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) {
                    if (keep_in && !keep_in[k]) continue;
                    int64_t u = in_src[k];
                    for (int64_t j = 0; j < d_in; j++) a[j] += or_load(H, h_dtype, u * d_in + j);
                    m++;
                }
                if (m > 0)
                    for (int64_t j = 0; j < d_in; j++) a[j] = a[j] / (double)m;
                for (int64_t j = 0; j < d_in; j++) a[d_in + j] = or_load(H, h_dtype, v * d_in + j);
            } else if (agg == 1) {
                int64_t m = 0;
                for (int64_t k = in_off[v]; k < in_off[v + 1]; k++)
                    if (!keep_in || keep_in[k]) m++;
                double din_hat = (double)m + 1.0;
                for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) {
                    if (keep_in && !keep_in[k]) continue;
                    int64_t u = in_src[k];
                    double c = 1.0 / sqrt(((double)deg_out[u] + 1.0) * din_hat);
                    for (int64_t j = 0; j < d_in; j++) a[j] += c * or_load(H, h_dtype, u * d_in + j);
                }
                double cs = 1.0 / sqrt(((double)deg_out[v] + 1.0) * din_hat);
                for (int64_t j = 0; j < d_in; j++) a[j] += cs * or_load(H, h_dtype, v * d_in + j);
            } else {
                for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) {
                    if (keep_in && !keep_in[k]) continue;
                    int64_t u = in_src[k];
                    for (int64_t j = 0; j < d_in; j++) a[j] += or_load(H, h_dtype, u * d_in + j);
                }
                for (int64_t j = 0; j < d_in; j++) a[j] += or_load(H, h_dtype, v * d_in + j);
            }
            for (int64_t o = 0; o < d_out; o++) {
                double z = bias ? bias[o] : 0.0;
                for (int64_t j = 0; j < cols; j++) z += W[o * cols + j] * a[j];
                if (relu && z < 0.0) z = 0.0;
                out[i * d_out + o] = z;
            }
        }
        free(a);
    }
    return bad ? -3 : 0;
}

/*
 * GINConv with a two-layer perceptron as its apply function and eps = 0
 * (Sec. 4.1 evaluates GINConv; the perceptron is the standard GIN update):
 *     a    = h_v + sum_{u in M(v)} h_u                    (sum aggregation)
 *     t    = ReLU(W1 a + b1)                              (W1: d_h x d_in)
 *     z    = W2 t + b2                                    (W2: d_out x d_h)
 * Output: out[i][j] = ReLU(z_j) if relu else z_j, for v = dst_ids[i] (all
 * vertices when dst_ids is NULL).  keep_in selects the propagated in-edges
 * (NULL = all).  b1, b2 may be NULL (zero).  Returns 0, or -3 when out of
 * memory.
 */
int or_gin_mlp_layer(int64_t n, const int64_t* in_off, const int32_t* in_src, const uint8_t* keep_in,
                     const void* H, int h_dtype, int64_t d_in, const double* W1, const double* b1, int64_t d_h,
                     const double* W2, const double* b2, int64_t d_out, int relu, int64_t n_dst,
                     const int64_t* dst_ids, double* out) {
    int64_t count = dst_ids ? n_dst : n;
    int bad = 0;
#pragma omp parallel
    {
        double* a = (double*)malloc((size_t)(d_in + d_h) * sizeof(double));
        double* t = a ? a + d_in : NULL;
        if (!a) bad = 1;
#pragma omp for schedule(dynamic, 256)
        for (int64_t i = 0; i < count; i++) {
            if (!a) continue;
            int64_t v = dst_ids ? dst_ids[i] : i;
            for (int64_t j = 0; j < d_in; j++) a[j] = or_load(H, h_dtype, v * d_in + j);
            for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) {
                if (keep_in && !keep_in[k]) continue;
                int64_t u = in_src[k];
                for (int64_t j = 0; j < d_in; j++) a[j] += or_load(H, h_dtype, u * d_in + j);
            }
            for (int64_t h = 0; h < d_h; h++) {
                double x = b1 ? b1[h] : 0.0;
                for (int64_t j = 0; j < d_in; j++) x += W1[h * d_in + j] * a[j];
                t[h] = x > 0.0 ? x : 0.0;
            }
            for (int64_t o = 0; o < d_out; o++) {
                double z = b2 ? b2[o] : 0.0;
                for (int64_t h = 0; h < d_h; h++) z += W2[o * d_h + h] * t[h];
                if (relu && z < 0.0) z = 0.0;
                out[i * d_out + o] = z;
            }
        }
        free(a);
    }
    return bad ? -3 : 0;
}

/*
 * GATConv, single head (Sec. 3.9, GATConv; Sec. 4.1 evaluates it):
 *     h'_u    = W h_u                                   (W: d_out x d_in)
 *     e_uv    = LeakyReLU(a^T [h'_u || h'_v])           (a = [a_src ; a_dst])
 *     alpha_uv = softmax over u in N-(v) of e_uv
 *     z_v     = sum_u alpha_uv h'_u + b,  out = ReLU(z) if relu.
 * N-(v) holds v's propagated in-neighbours and v itself (every vertex
 * aggregates a self message); keep_in selects the propagated in-edges (NULL
 * = all).  attn = [a_src (d_out) | a_dst (d_out)]; slope = LeakyReLU's
 * negative slope.  The softmax subtracts the neighbourhood's largest score
 * (the same value in exact arithmetic).  h' is computed for every vertex.
 * Returns 0, or -3 when out of memory.
 */
int or_gat_layer(int64_t n, const int64_t* in_off, const int32_t* in_src, const uint8_t* keep_in,
                 const void* H, int h_dtype, int64_t d_in, const double* W, const double* attn,
                 const double* bias, int64_t d_out, int relu, double slope, int64_t n_dst,
                 const int64_t* dst_ids, double* out) {
    double* hp = (double*)malloc((size_t)(n > 0 ? n : 1) * (size_t)d_out * sizeof(double));
    double* sc = (double*)malloc((size_t)(n > 0 ? n : 1) * 2 * sizeof(double));
    if (!hp || !sc) return -3;
#pragma omp parallel for schedule(dynamic, 256)
    for (int64_t u = 0; u < n; u++) {
        double s_src = 0.0, s_dst = 0.0;
        for (int64_t o = 0; o < d_out; o++) {
            double z = 0.0;
            for (int64_t j = 0; j < d_in; j++) z += W[o * d_in + j] * or_load(H, h_dtype, u * d_in + j);
            hp[u * d_out + o] = z;
            s_src += attn[o] * z;
            s_dst += attn[d_out + o] * z;
        }
        sc[2 * u] = s_src;
        sc[2 * u + 1] = s_dst;
    }
    int64_t count = dst_ids ? n_dst : n;
    int bad = 0;
#pragma omp parallel
    {
        double* a = (double*)malloc((size_t)d_out * sizeof(double));
        if (!a) bad = 1;
#pragma omp for schedule(dynamic, 256)
        for (int64_t i = 0; i < count; i++) {
            if (!a) continue;
            int64_t v = dst_ids ? dst_ids[i] : i;
            double tv = sc[2 * v + 1];
            /* the largest score: the self message first, then the kept in-edges */
            double e = sc[2 * v] + tv;
            double m = e > 0.0 ? e : slope * e;
            for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) {
                if (keep_in && !keep_in[k]) continue;
                e = sc[2 * (int64_t)in_src[k]] + tv;
                e = e > 0.0 ? e : slope * e;
                if (e > m) m = e;
            }
            /* unnormalised weights exp(e - m), their sum, and the weighted rows */
            for (int64_t o = 0; o < d_out; o++) a[o] = 0.0;
            double ssum = 0.0;
            for (int64_t k = in_off[v] - 1; k < in_off[v + 1]; k++) {
                int64_t u;
                if (k < in_off[v]) {
                    u = v;
                } else {
                    if (keep_in && !keep_in[k]) continue;
                    u = in_src[k];
                }
                e = sc[2 * u] + tv;
                e = e > 0.0 ? e : slope * e;
                double w = exp(e - m);
                ssum += w;
                for (int64_t o = 0; o < d_out; o++) a[o] += w * hp[u * d_out + o];
            }
            for (int64_t o = 0; o < d_out; o++) {
                double z = a[o] / ssum + (bias ? bias[o] : 0.0);
                if (relu) z = z < 0.0 ? 0.0 : z;
                out[i * d_out + o] = z;
            }
        }
        free(a);
    }
    free(hp);
    free(sc);
    return bad ? -3 : 0;
}

/* ------------------------------------------------------------ reorder ---- */
/*
 * Degree/BFS vertex ordering: a reading of a degree-sorted breadth-first
 * ordering as the cheap topology-aware bootstrap (the paper bootstraps with
 * RCMK and refines with its Algorithm 1, Sec. 3.8; see or_reorder_ta).
 *
 *   - root order: all vertices by (in-degree descending, ID ascending);
 *   - each root not yet visited starts a breadth-first search over IN-edges
 *     (from a vertex to its in-neighbours, i.e. its message sources), so a
 *     destination's sources receive consecutive ranks;
 *   - a dequeued vertex appends its unvisited in-neighbours in
 *     (in-degree descending, ID ascending) order;
 *   - new_of_old[v] = position of v in the visit order.
 * The order is unique, so results are compared bit for bit.
 */
static const int32_t* g_or_deg;
static int or_rank_cmp(const void* x, const void* y) {
    int32_t a = *(const int32_t*)x, b = *(const int32_t*)y;
    if (g_or_deg[a] != g_or_deg[b]) return g_or_deg[a] > g_or_deg[b] ? -1 : 1;
    return (a > b) - (a < b);
}
int or_reorder_bfs(int64_t n, const int64_t* in_off, const int32_t* in_src, int32_t* new_of_old) {
    int32_t* deg = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    int32_t* order = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    int32_t* queue = (int32_t*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int32_t));
    uint8_t* seen = (uint8_t*)calloc((size_t)(n > 0 ? n : 1), 1);
    int64_t maxd = 0;
    for (int64_t v = 0; v < n; v++) {
        deg[v] = (int32_t)(in_off[v + 1] - in_off[v]);
        if (deg[v] > maxd) maxd = deg[v];
        order[v] = (int32_t)v;
    }
    int32_t* kids = (int32_t*)malloc((size_t)(maxd > 0 ? maxd : 1) * sizeof(int32_t));
    if (!deg || !order || !queue || !seen || !kids) return -3;
    g_or_deg = deg;
    qsort(order, (size_t)n, sizeof(int32_t), or_rank_cmp);
    int64_t head = 0, tail = 0;
    for (int64_t r = 0; r < n; r++) {
        int32_t root = order[r];
        if (seen[root]) continue;
        seen[root] = 1;
        queue[tail++] = root;
        while (head < tail) {
            int32_t x = queue[head++];
            int64_t nk = 0;
            for (int64_t k = in_off[x]; k < in_off[x + 1]; k++) {
                int32_t w = in_src[k];
                if (!seen[w]) { seen[w] = 1; kids[nk++] = w; }
            }
            qsort(kids, (size_t)nk, sizeof(int32_t), or_rank_cmp);
            for (int64_t j = 0; j < nk; j++) queue[tail++] = kids[j];
        }
    }
    for (int64_t i = 0; i < n; i++) new_of_old[queue[i]] = (int32_t)i;
    free(deg); free(order); free(queue); free(seen); free(kids);
    return 0;
}

/*
 * RCMK: reverse Cuthill-McKee, the bandwidth-reducing bootstrap the paper
 * applies before Alg. 1 (Sec. 3.8 cites Chan and George's linear-time
 * formulation).  It works on the symmetrised graph: S(v) = the distinct
 * vertices u != v with (u, v) or (v, u) an edge, and delta(v) = |S(v)|.
 *   - roots: every vertex in (delta ascending, ID ascending) order; each one
 *     not yet visited starts a breadth-first search;
 *   - a dequeued vertex appends its unvisited neighbours in S in the same
 *     (delta ascending, ID ascending) order (Cuthill-McKee);
 *   - the visit order is reversed: new_of_old[v] = n - 1 - position of v.
 * Readings taken here: no pseudo-peripheral root search (the minimum degree
 * vertex of each component starts it) and ties by the lower ID, so the order
 * is unique and compared bit for bit.  Returns 0, or -3 when out of memory.
 */
static const int32_t* g_or_sdeg;
static int or_cm_cmp(const void* x, const void* y) {
    int32_t a = *(const int32_t*)x, b = *(const int32_t*)y;
    if (g_or_sdeg[a] != g_or_sdeg[b]) return g_or_sdeg[a] < g_or_sdeg[b] ? -1 : 1;
    return (a > b) - (a < b);
}
int or_reorder_rcm(int64_t n, const int64_t* row_off, const int32_t* col_dst, const int64_t* in_off,
                   const int32_t* in_src, int32_t* new_of_old) {
    size_t nn = (size_t)(n > 0 ? n : 1);
    int64_t cap = row_off[n] + in_off[n];
    int32_t* adj = (int32_t*)malloc((size_t)(cap > 0 ? cap : 1) * sizeof(int32_t));
    int32_t* deg = (int32_t*)malloc(nn * sizeof(int32_t));
    int32_t* order = (int32_t*)malloc(nn * sizeof(int32_t));
    int32_t* queue = (int32_t*)malloc(nn * sizeof(int32_t));
    int64_t* count = (int64_t*)calloc(nn + 1, sizeof(int64_t));
    uint8_t* seen = (uint8_t*)calloc(nn, 1);
    if (!adj || !deg || !order || !queue || !count || !seen) return -3;
    /* S(v): out- and in-neighbours together, sorted, repeats dropped; v's
     * list starts at row_off[v] + in_off[v] */
#pragma omp parallel for schedule(dynamic, 1024)
    for (int64_t v = 0; v < n; v++) {
        int32_t* a = adj + row_off[v] + in_off[v];
        int64_t k = 0;
        for (int64_t i = row_off[v]; i < row_off[v + 1]; i++) a[k++] = col_dst[i];
        for (int64_t i = in_off[v]; i < in_off[v + 1]; i++) a[k++] = in_src[i];
        qsort(a, (size_t)k, sizeof(int32_t), or_i32_cmp);
        int64_t m = 0;
        for (int64_t i = 0; i < k; i++)
            if (a[i] != v && (m == 0 || a[i] != a[m - 1])) a[m++] = a[i];
        deg[v] = (int32_t)m;
    }
    if (n >= (1 << 24)) fprintf(stderr, "reorder_rcm: symmetric lists done\n");
    /* root order: a counting sort by delta keeps IDs ascending within a degree */
    for (int64_t v = 0; v < n; v++) count[deg[v] + 1]++;
    for (int64_t d = 0; d < n; d++) count[d + 1] += count[d];
    for (int64_t v = 0; v < n; v++) order[count[deg[v]]++] = (int32_t)v;
    g_or_sdeg = deg;
    int64_t head = 0, tail = 0;
    for (int64_t r = 0; r < n; r++) {
        int32_t root = order[r];
        if (seen[root]) continue;
        seen[root] = 1;
        queue[tail++] = root;
        while (head < tail) {
            int32_t x = queue[head++];
            const int32_t* a = adj + row_off[x] + in_off[x];
            int64_t first = tail;
            for (int64_t i = 0; i < deg[x]; i++)
                if (!seen[a[i]]) { seen[a[i]] = 1; queue[tail++] = a[i]; }
            qsort(queue + first, (size_t)(tail - first), sizeof(int32_t), or_cm_cmp);
        }
    }
    for (int64_t i = 0; i < n; i++) new_of_old[queue[i]] = (int32_t)(n - 1 - i);
    free(adj); free(deg); free(order); free(queue); free(count); free(seen);
    return 0;
}

/*
 * Total span C(pi) = sum_v (max_{u in N-(v)} pi(u) - min_{u in N-(v)} pi(u))
 * (Sec. 3.8).  N-(v) holds v's in-neighbours and v itself: every vertex
 * aggregates a self message, and a vertex with only that message has span 0,
 * so a vertex's residency runs from its first to its last message, the self
 * message included.
 */
int64_t or_total_span(int64_t n, const int64_t* in_off, const int32_t* in_src, const int32_t* pi) {
    int64_t total = 0;
#pragma omp parallel for reduction(+ : total) schedule(dynamic, 4096)
    for (int64_t v = 0; v < n; v++) {
        int64_t lo = pi[v], hi = pi[v];
        for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) {
            int64_t p = pi[in_src[k]];
            if (p < lo) lo = p;
            if (p > hi) hi = p;
        }
        total += hi - lo;
    }
    return total;
}

/*
 * Residency profile at chunk granularity (Sec. 3.8's A(t), with t counted in
 * chunks of `chunk` consecutive ranks): with N-(v) including v,
 *     a(v) = min_{u in N-(v)} floor(pi(u) / chunk),  c(v) = max likewise,
 *     A[k] = #{v : a(v) <= k < c(v)},  k = 0 .. ceil(n / chunk) - 1,
 * the destinations holding a partial state after chunk k.  With chunk = 1,
 * sum_k A[k] = C(pi) (the paper's identity M = C(pi)).
 */
void or_active_profile(int64_t n, const int64_t* in_off, const int32_t* in_src, const int32_t* pi, int64_t chunk,
                       int64_t* A) {
    int64_t nch = (n + chunk - 1) / chunk;
    int64_t* diff = (int64_t*)calloc((size_t)nch + 1, sizeof(int64_t));
#pragma omp parallel for schedule(dynamic, 4096)
    for (int64_t v = 0; v < n; v++) {
        int64_t lo = pi[v] / chunk, hi = lo;
        for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) {
            int64_t c = pi[in_src[k]] / chunk;
            if (c < lo) lo = c;
            if (c > hi) hi = c;
        }
        if (hi > lo) {
#pragma omp atomic
            diff[lo] += 1;
#pragma omp atomic
            diff[hi] -= 1;
        }
    }
    int64_t run = 0;
    for (int64_t k = 0; k < nch; k++) { run += diff[k]; A[k] = run; }
    free(diff);
}

/*
 * The residency protocol of a budgeted layer (Sec. 3.5), simulated at the
 * level of slots: which partial states are evicted and reloaded, chunk by
 * chunk, for a pool of S rows of which H hold hubs.  Chunks of `chunk`
 * consecutive sources run in ascending order.  keep (per CSR edge, NULL =
 * every edge) marks the propagated edges; M(v) = v's propagated in-edges.
 *   - hubs: the H vertices first by (|M(v)| descending, ID ascending); their
 *     rows never move;
 *   - pending(v) starts at |M(v)| + 1 (the self message arrives in v's own
 *     chunk);
 *   - before chunk k: its touched vertices (destinations of its propagated
 *     edges, and its own vertices) that hold no row ask for one; if the free
 *     rows fall short by M, the M candidates (holding a row, not hubs, not
 *     touched by chunk k, still pending) with the smallest (key, ID) are
 *     evicted.  Keys (Sec. 3.5.3 and the policies of the eviction study):
 *       0 fewest pending: pending(v), the exact count of messages due;
 *       1 random: H(seed, 7, k, v) >> 50;
 *       2 FIFO: the chunk at which v last took a row;
 *       3 LRU: the last chunk that touched v;
 *   - the asking vertices take rows (an evicted one is reloaded), the chunk's
 *     messages arrive, and touched vertices that completed free their rows.
 * Outputs the eviction and reload totals and reloads per vertex.  Returns 0,
 * -6 when the candidates cannot free enough rows, -3 when out of memory.
 */
static const int32_t* g_or_m;
static int or_hub_cmp(const void* x, const void* y) {
    int32_t a = *(const int32_t*)x, b = *(const int32_t*)y;
    if (g_or_m[a] != g_or_m[b]) return g_or_m[a] > g_or_m[b] ? -1 : 1;
    return (a > b) - (a < b);
}
typedef struct { int64_t key; int32_t v; } or_victim;
static int or_victim_cmp(const void* x, const void* y) {
    const or_victim* a = (const or_victim*)x; const or_victim* b = (const or_victim*)y;
    if (a->key != b->key) return a->key < b->key ? -1 : 1;
    return (a->v > b->v) - (a->v < b->v);
}
int or_residency_sim(int64_t n, const int64_t* row_off, const int32_t* col_dst, const uint8_t* keep, int64_t chunk,
                     int64_t S, int64_t H, int policy, uint64_t seed, int64_t* evictions, int64_t* reloads,
                     int32_t* reloads_of) {
    size_t nn = (size_t)(n > 0 ? n : 1);
    int32_t* m = (int32_t*)calloc(nn, sizeof(int32_t));
    int32_t* order = (int32_t*)malloc(nn * sizeof(int32_t));
    int64_t* pend = (int64_t*)malloc(nn * sizeof(int64_t));
    int32_t* mark = (int32_t*)malloc(nn * sizeof(int32_t));
    int32_t* adm = (int32_t*)calloc(nn, sizeof(int32_t));
    uint8_t* hub = (uint8_t*)calloc(nn, 1);
    uint8_t* resident = (uint8_t*)calloc(nn, 1);
    uint8_t* evicted = (uint8_t*)calloc(nn, 1);
    int32_t* touched = (int32_t*)malloc(nn * sizeof(int32_t));
    int32_t* need = (int32_t*)malloc(nn * sizeof(int32_t));
    or_victim* cand = (or_victim*)malloc(nn * sizeof(or_victim));
    if (!m || !order || !pend || !mark || !adm || !hub || !resident || !evicted || !touched || !need || !cand)
        return -3;
    for (int64_t u = 0; u < n; u++)
        for (int64_t i = row_off[u]; i < row_off[u + 1]; i++)
            if (!keep || keep[i]) m[col_dst[i]]++;
    for (int64_t v = 0; v < n; v++) {
        order[v] = (int32_t)v;
        pend[v] = (int64_t)m[v] + 1;
        mark[v] = -1;
        reloads_of[v] = 0;
    }
    g_or_m = m;
    qsort(order, nn, sizeof(int32_t), or_hub_cmp);
    for (int64_t j = 0; j < H && j < n; j++) { hub[order[j]] = 1; resident[order[j]] = 1; }
    int64_t free_rows = S - H;
    *evictions = 0;
    *reloads = 0;
    int rc = free_rows < 0 ? -6 : 0;
    int64_t nch = (n + chunk - 1) / chunk;
    for (int64_t k = 0; k < nch && rc == 0; k++) {
        int64_t b = k * chunk, e = b + chunk < n ? b + chunk : n;
        int64_t nt = 0, nq = 0;
        for (int64_t u = b; u < e; u++)
            for (int64_t i = row_off[u]; i < row_off[u + 1]; i++) {
                int32_t v = col_dst[i];
                if ((!keep || keep[i]) && mark[v] != (int32_t)k) { mark[v] = (int32_t)k; touched[nt++] = v; }
            }
        for (int64_t v = b; v < e; v++)
            if (mark[v] != (int32_t)k) { mark[v] = (int32_t)k; touched[nt++] = (int32_t)v; }
        /* the LRU key needs each candidate's last touch before chunk k: the
         * candidates are exactly the vertices chunk k does not touch, so
         * their marks still hold it */
        for (int64_t t = 0; t < nt; t++)
            if (pend[touched[t]] > 0 && !resident[touched[t]]) need[nq++] = touched[t];
        if (nq > free_rows) {
            int64_t M = nq - free_rows, nc = 0;
            for (int64_t v = 0; v < n; v++) {
                if (!resident[v] || hub[v] || mark[v] == (int32_t)k || pend[v] <= 0) continue;
                int64_t key;
                if (policy == 1) {
                    uint64_t args[2] = {(uint64_t)k, (uint64_t)v};
                    key = (int64_t)(or_hash(seed, 7, 2, args) >> 50);
                } else if (policy == 2) {
                    key = adm[v];
                } else if (policy == 3) {
                    key = mark[v];
                } else {
                    key = pend[v];
                }
                cand[nc].key = key;
                cand[nc].v = (int32_t)v;
                nc++;
            }
            if (nc < M) { rc = -6; break; }
            qsort(cand, (size_t)nc, sizeof(or_victim), or_victim_cmp);
            for (int64_t j = 0; j < M; j++) { resident[cand[j].v] = 0; evicted[cand[j].v] = 1; }
            free_rows += M;
            *evictions += M;
        }
        for (int64_t j = 0; j < nq; j++) {
            int32_t v = need[j];
            resident[v] = 1;
            adm[v] = (int32_t)k;
            if (evicted[v]) { evicted[v] = 0; reloads_of[v]++; (*reloads)++; }
        }
        free_rows -= nq;
        for (int64_t u = b; u < e; u++)
            for (int64_t i = row_off[u]; i < row_off[u + 1]; i++)
                if (!keep || keep[i]) pend[col_dst[i]]--;
        for (int64_t v = b; v < e; v++) pend[v]--;
        for (int64_t t = 0; t < nt; t++) {
            int32_t v = touched[t];
            if (pend[v] == 0 && !hub[v] && resident[v]) { resident[v] = 0; free_rows++; }
        }
    }
    free(m); free(order); free(pend); free(mark); free(adm); free(hub); free(resident); free(evicted);
    free(touched); free(need); free(cand);
    return rc;
}

/* ------------------------------------- topology-aware reordering (Alg. 1) -- */
/*
 * Sec. 3.8 minimises the in-neighbourhood dispersion
 *     J(r, mu) = sum_v 1/d(v) sum_{u in N(v)} (r(u) - mu(v))^2
 * over real positions r by alternating its two closed-form minimisers
 *     mu*(v) = (1/d(v)) sum_{u in N(v)} r(u)                      (Eq. for mu*)
 *     r*(w)  = sum_{v : w in N(v)} mu(v)/d(v) / sum_{v : w in N(v)} 1/d(v)
 * and ranks the vertices by r (Alg. 1).  N(v) holds v's propagated
 * in-neighbours and v itself -- every vertex aggregates a self message, so
 * d(v) = d_in(v) + 1 >= 1 -- hence {v : w in N(v)} = {w} and w's
 * out-neighbours.  Every sum is taken in fp64, the self term first and then
 * the neighbours in ascending ID; ArgSort breaks ties by the lower vertex ID.
 *
 * One update: r_in -> mu -> r_out (CSR for the out-neighbours, in-lists for
 * the in-neighbours).
 */
void or_ta_step(int64_t n, const int64_t* row_off, const int32_t* col_dst, const int64_t* in_off,
                const int32_t* in_src, const double* r_in, double* mu, double* r_out) {
#pragma omp parallel for schedule(dynamic, 1024)
    for (int64_t v = 0; v < n; v++) {
        double s = r_in[v];
        for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) s += r_in[in_src[k]];
        mu[v] = s / (double)(in_off[v + 1] - in_off[v] + 1);
    }
#pragma omp parallel for schedule(dynamic, 1024)
    for (int64_t w = 0; w < n; w++) {
        double d = (double)(in_off[w + 1] - in_off[w] + 1);
        double num = mu[w] / d, den = 1.0 / d;
        for (int64_t i = row_off[w]; i < row_off[w + 1]; i++) {
            int32_t v = col_dst[i];
            double dv = (double)(in_off[v + 1] - in_off[v] + 1);
            num += mu[v] / dv;
            den += 1.0 / dv;
        }
        r_out[w] = num / den;
    }
}

typedef struct { double r; int32_t v; } or_pos;
static int or_pos_cmp(const void* x, const void* y) {
    const or_pos* a = (const or_pos*)x; const or_pos* b = (const or_pos*)y;
    if (a->r != b->r) return a->r < b->r ? -1 : 1;
    return (a->v > b->v) - (a->v < b->v);
}

/*
 * The dispersion J of Sec. 3.8 for positions x, at the centres that
 * minimise it for those positions:
 *     mu(v) = (1/d(v)) sum_{u in N(v)} x(u),
 *     J     = sum_v 1/d(v) sum_{u in N(v)} (x(u) - mu(v))^2,
 * N(v) = v and its propagated in-neighbours (the self message), d(v) = |N(v)|.
 * Two plain passes per vertex (centre, then squared deviations), fp64.
 * Called with x = the ranks of an ordering, this is the J of that ordering.
 */
double or_dispersion(int64_t n, const int64_t* in_off, const int32_t* in_src, const double* x) {
    double total = 0.0;
#pragma omp parallel for reduction(+ : total) schedule(dynamic, 4096)
    for (int64_t v = 0; v < n; v++) {
        double d = (double)(in_off[v + 1] - in_off[v] + 1);
        double s = x[v];
        for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) s += x[in_src[k]];
        double mu = s / d;
        double q = (x[v] - mu) * (x[v] - mu);
        for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) q += (x[in_src[k]] - mu) * (x[in_src[k]] - mu);
        total += q / d;
    }
    return total;
}

/*
 * Alg. 1 (Sec. 3.8) from the bootstrap order pi0 (new ID of each vertex;
 * NULL = identity).  The real positions are initialised once, r(v) = pi0(v);
 * each update then
 *     1. sets the centres mu = mu*(r) from the current positions,
 *     2. sets the positions r = r*(mu) from those centres,
 *     3. ranks the positions, pi = ArgSort(r), ties by the lower vertex ID,
 * and the loop ends once an update leaves pi unchanged (pi has converged) or
 * after `iters` updates.  The positions r are carried from one update to the
 * next; the ranks are only read off them.
 * Outputs: pi_out (int32[n]); r_out (double[n] or NULL): the positions after
 * the last update made (pi0 when none); spans[t] (or NULL) = C(pi_t), with
 * pi_0 the bootstrap (or_total_span); disp[t] (or NULL) = J of the ordering
 * pi_t, its ranks taken as positions (or_dispersion); *done = updates made.
 * Returns 0, or -3 when out of memory.
 */
int or_reorder_ta(int64_t n, const int64_t* row_off, const int32_t* col_dst, const int64_t* in_off,
                  const int32_t* in_src, const int32_t* pi0, int iters, int32_t* pi_out, double* r_out,
                  int64_t* spans, double* disp, int* done) {
    size_t nn = (size_t)(n > 0 ? n : 1);
    double* r = (double*)malloc(nn * sizeof(double));
    double* r2 = (double*)malloc(nn * sizeof(double));
    double* mu = (double*)malloc(nn * sizeof(double));
    double* rank = (double*)malloc(nn * sizeof(double));
    or_pos* pos = (or_pos*)malloc(nn * sizeof(or_pos));
    if (!r || !r2 || !mu || !rank || !pos) { free(r); free(r2); free(mu); free(rank); free(pos); return -3; }
    for (int64_t v = 0; v < n; v++) {
        pi_out[v] = pi0 ? pi0[v] : (int32_t)v;
        r[v] = (double)pi_out[v];
        rank[v] = r[v];
    }
    if (spans) spans[0] = or_total_span(n, in_off, in_src, pi_out);
    if (disp) disp[0] = or_dispersion(n, in_off, in_src, rank);
    *done = 0;
    for (int t = 1; t <= iters; t++) {
        or_ta_step(n, row_off, col_dst, in_off, in_src, r, mu, r2);
        memcpy(r, r2, nn * sizeof(double));
        for (int64_t v = 0; v < n; v++) { pos[v].r = r[v]; pos[v].v = (int32_t)v; }
        qsort(pos, (size_t)n, sizeof(or_pos), or_pos_cmp);
        int changed = 0;
        for (int64_t k = 0; k < n; k++) {
            if (pi_out[pos[k].v] != (int32_t)k) changed = 1;
            pi_out[pos[k].v] = (int32_t)k;
            rank[pos[k].v] = (double)k;
        }
        *done = t;
        if (spans) spans[t] = or_total_span(n, in_off, in_src, pi_out);
        if (disp) disp[t] = or_dispersion(n, in_off, in_src, rank);
        if (n >= (1 << 24)) fprintf(stderr, "reorder_ta: update %d of %d done\n", t, iters);
        if (!changed) break;
    }
    if (r_out) memcpy(r_out, r, (size_t)n * sizeof(double));
    free(r); free(r2); free(mu); free(rank); free(pos);
    return 0;
}
