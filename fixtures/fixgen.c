/*
 * Seeded synthetic inputs for the layer-wise broadcast GNN inference path.
 *
 * This module produces INPUTS only: RMAT edge lists, vertex features, layer
 * weights and biases, and the random-ID relabelling used for the skewed
 * graph workload.  It holds none of the method's arithmetic (no aggregation,
 * no normalisation, no sampling, no reordering) and is the one piece of code
 * that both the CPU oracle and the GPU library see: the two consume the same
 * bytes that it writes.
 *
 * Counter-based generator.  Every random number is a pure function of the
 * seed and of integer coordinates:
 *     H(s, t, x1, ..., xk):  h = s;  for x in (t, x1, ..., xk): h = mix64(h + G + x)
 * where mix64 is the SplitMix64 output finaliser and G = 0x9e3779b97f4a7c15
 * its golden-ratio increment (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014).  H(0, 0) is therefore the
 * first output of SplitMix64 started from state 0.
 *
 * Tags: 1 RMAT, 2 features, 3 weights, 5 random vertex IDs, 6 bias.
 * (Tag 4 is reserved for the fanout sampler, which is method code and lives
 * with each implementation of the method, not here.)
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>
#include <stdio.h>

#define FX_GAMMA 0x9e3779b97f4a7c15ULL

static inline uint64_t fx_mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}
static inline uint64_t fx_step(uint64_t h, uint64_t x) { return fx_mix64(h + FX_GAMMA + x); }

uint64_t fx_hash(uint64_t seed, uint64_t tag, int nargs, const uint64_t* args) {
    uint64_t h = fx_step(seed, tag);
    for (int i = 0; i < nargs; i++) h = fx_step(h, args[i]);
    return h;
}

/* ---------------------------------------------------------------- RMAT ---- */
/*
 * Edge set = the first `e` distinct valid pairs in attempt order.
 * Attempt j draws one 53-bit uniform per level b (MSB first) from
 * H(seed, 1, j, b) >> 11 and picks quadrant (0,0), (0,1), (1,0), (1,1) of the
 * adjacency matrix with probabilities a, b, c, 1-a-b-c, setting one bit of
 * (u, v) per level.  Pairs with u >= n, v >= n or u == v are rejected, as are
 * pairs already accepted.  No noise is added.
 *
 * Parallel but deterministic: attempts are drawn in batches; duplicate
 * detection is partitioned by a hash of the pair so that each thread owns a
 * disjoint hash-set shard and walks the batch in attempt order.
 */
typedef struct { uint64_t* slots; uint64_t mask; int64_t used; } fx_set;

static int fx_set_insert(fx_set* s, uint64_t key) { /* key != 0; 1 if new */
    uint64_t i = fx_mix64(key) & s->mask;
    for (;;) {
        uint64_t k = s->slots[i];
        if (k == 0) { s->slots[i] = key; s->used++; return 1; }
        if (k == key) return 0;
        i = (i + 1) & s->mask;
    }
}

int64_t fx_rmat(uint64_t seed, int64_t n, int64_t e, double a, double b, double c,
                int32_t* src, int32_t* dst) {
    if (n < 2 || e < 0) return -1;
    if ((double)e > (double)n * (double)(n - 1)) return -1;
    int scale = 0;
    while (((int64_t)1 << scale) < n) scale++;
    const uint64_t two53 = (uint64_t)1 << 53;
    const uint64_t ta = (uint64_t)(a * (double)two53);
    const uint64_t tb = (uint64_t)((a + b) * (double)two53);
    const uint64_t tc = (uint64_t)((a + b + c) * (double)two53);

    int nthr = omp_get_max_threads();
    if (nthr < 1) nthr = 1;
    /* shard capacity: ~2x the expected share of e, power of two */
    uint64_t per = (uint64_t)(e / nthr + 1) * 2 + 1024;
    uint64_t cap = 1;
    while (cap < per) cap <<= 1;
    fx_set* sets = (fx_set*)calloc((size_t)nthr, sizeof(fx_set));
    for (int t = 0; t < nthr; t++) {
        sets[t].slots = (uint64_t*)calloc(cap, sizeof(uint64_t));
        sets[t].mask = cap - 1;
        if (!sets[t].slots) return -2;
    }
    /* a batch never holds more attempts than edges still missing (plus a
     * small floor), so the shards never hold more than e + 1024 pairs */
    const int64_t max_batch = 1 << 22;
    uint64_t* cand = (uint64_t*)malloc((size_t)max_batch * sizeof(uint64_t));
    uint8_t* ok = (uint8_t*)malloc((size_t)max_batch);
    int64_t accepted = 0, attempt = 0;
    int err = 0;
    while (accepted < e && !err) {
        int64_t batch = e - accepted;
        if (batch < 1024) batch = 1024;
        if (batch > max_batch) batch = max_batch;
        /* draw a batch of attempts; 0 marks a rejected attempt */
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < batch; i++) {
            uint64_t j = (uint64_t)(attempt + i);
            uint64_t u = 0, v = 0;
            uint64_t h0 = fx_step(fx_step(seed, 1), j);
            for (int lv = 0; lv < scale; lv++) {
                uint64_t r = fx_step(h0, (uint64_t)lv) >> 11;
                uint64_t ub, vb;
                if (r < ta) { ub = 0; vb = 0; }
                else if (r < tb) { ub = 0; vb = 1; }
                else if (r < tc) { ub = 1; vb = 0; }
                else { ub = 1; vb = 1; }
                u = (u << 1) | ub;
                v = (v << 1) | vb;
            }
            int valid = (u < (uint64_t)n) && (v < (uint64_t)n) && (u != v);
            cand[i] = valid ? ((u << 32) | v) + 1 : 0;
        }
        /* shard-owned duplicate detection in attempt order */
#pragma omp parallel num_threads(nthr)
        {
            int t = omp_get_thread_num();
            fx_set* s = &sets[t];
            for (int64_t i = 0; i < batch; i++) {
                uint64_t k = cand[i];
                if (k == 0) { if (t == 0) ok[i] = 0; continue; }
                if ((int)(fx_mix64(k ^ 0x5bd1e995ULL) % (uint64_t)nthr) != t) continue;
                if ((uint64_t)s->used * 10 > cap * 8) { ok[i] = 0; err = 1; continue; }
                ok[i] = (uint8_t)fx_set_insert(s, k);
            }
        }
        if (err) break;
        for (int64_t i = 0; i < batch && accepted < e; i++) {
            if (!ok[i]) continue;
            uint64_t k = cand[i] - 1;
            src[accepted] = (int32_t)(k >> 32);
            dst[accepted] = (int32_t)(k & 0xffffffffULL);
            accepted++;
        }
        attempt += batch;
        if (attempt > e * 64 + (int64_t)max_batch * 4) { err = 2; break; }
        /* large graphs take minutes: a progress line every 2^28 edges */
        if (e >= ((int64_t)1 << 28) && (accepted >> 28) != ((accepted - batch) >> 28) && accepted < e)
            fprintf(stderr, "rmat: %lld of %lld edges\n", (long long)accepted, (long long)e);
    }
    for (int t = 0; t < nthr; t++) free(sets[t].slots);
    free(sets); free(cand); free(ok);
    if (err) return -3;
    return attempt;
}

/* ----------------------------------------------------- precision casts ---- */
/* round-to-nearest-even conversions of fp32 to the 16-bit storage types */
static inline uint16_t fx_f32_to_bf16(float f) {
    uint32_t x; memcpy(&x, &f, 4);
    if ((x & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((x >> 16) | 0x40u);
    return (uint16_t)((x + 0x7fffu + ((x >> 16) & 1u)) >> 16);
}
static inline uint16_t fx_f32_to_f16(float f) {
    uint32_t x; memcpy(&x, &f, 4);
    uint32_t sign = (x >> 16) & 0x8000u, ax = x & 0x7fffffffu;
    if (ax >= 0x7f800000u) return (uint16_t)(sign | (ax > 0x7f800000u ? 0x7e00u : 0x7c00u));
    if (ax >= 0x477ff000u) return (uint16_t)(sign | 0x7c00u);
    if (ax < 0x38800000u) { /* fp16 subnormal range: scale by 2^24 is exact */
        float m; uint32_t mx = ax; memcpy(&m, &mx, 4);
        return (uint16_t)(sign | (uint32_t)nearbyintf(m * 16777216.0f));
    }
    uint32_t r = ax - 0x38000000u;
    r = (r + 0x0fffu + ((r >> 13) & 1u)) >> 13;
    return (uint16_t)(sign | r);
}

/* ------------------------------------------------------------ features ---- */
/*
 * Row v, column j.  dist 0: U[-1, 1) = ((H(seed,2,v,j) >> 40) * 2^-23) - 1,
 * exact in fp32.  dist 1: N(0,1) by the Box-Muller transform (Box and
 * Muller, 1958) in fp64 from u1 = ((H(seed,2,v,j,0) >> 11) + 1) * 2^-53 and
 * u2 = (H(seed,2,v,j,1) >> 11) * 2^-53, rounded fp64 -> fp32.  out_dtype
 * 0 fp32, 1 bf16, 2 fp16: the fp32 value is rounded (RNE) to the 16-bit type.
 * Writes rows [v0, v1) of width d into `out` (row-major, row stride d).
 */
static inline float fx_feature(uint64_t seed, int dist, uint64_t v, uint64_t j) {
    uint64_t h = fx_step(fx_step(fx_step(seed, 2), v), j);
    if (dist == 0) {
        return (float)((double)(h >> 40) * 0x1.0p-23 - 1.0);
    }
    uint64_t h0 = fx_step(h, 0), h1 = fx_step(h, 1);
    double u1 = ((double)(h0 >> 11) + 1.0) * 0x1.0p-53;
    double u2 = (double)(h1 >> 11) * 0x1.0p-53;
    double z = sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925286766559 * u2);
    return (float)z;
}

/*
 * One fp32 row of dist 0 from the row prefix hv = H(seed, 2, v): the same
 * values as fx_feature, written so that the compiler vectorises it (x =
 * top 24 bits; x * 2^-23 - 1 = (x - 2^23) * 2^-23 is exact in fp32).  A
 * copy built for AVX-512 (64-bit vector multiplies) is used where the host
 * has it.
 */
#define FX_UNIFORM_ROW_BODY                                                      \
    for (int64_t j = 0; j < d; j++) {                                            \
        uint64_t z = hv + FX_GAMMA + (uint64_t)j;                                \
        z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;                             \
        z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;                             \
        z ^= z >> 31;                                                            \
        row[j] = (float)((int32_t)(z >> 40) - 8388608) * 0x1.0p-23f;             \
    }
__attribute__((target("avx512f,avx512dq,avx512vl")))
static void fx_uniform_row_avx512(uint64_t hv, int64_t d, float* row) { FX_UNIFORM_ROW_BODY }
static void fx_uniform_row_plain(uint64_t hv, int64_t d, float* row) { FX_UNIFORM_ROW_BODY }
static void fx_uniform_row(uint64_t hv, int64_t d, float* row) {
    static int wide = -1;
    if (wide < 0) wide = __builtin_cpu_supports("avx512dq") && __builtin_cpu_supports("avx512vl") ? 1 : 0;
    if (wide) fx_uniform_row_avx512(hv, d, row);
    else fx_uniform_row_plain(hv, d, row);
}

void fx_features(uint64_t seed, int dist, int64_t v0, int64_t v1, int64_t d, int out_dtype, void* out) {
    const uint64_t s2 = fx_step(seed, 2);
#pragma omp parallel for schedule(static)
    for (int64_t v = v0; v < v1; v++) {
        if (dist == 0 && out_dtype == 0) {
            fx_uniform_row(fx_step(s2, (uint64_t)v), d, (float*)out + (v - v0) * d);
            continue;
        }
        for (int64_t j = 0; j < d; j++) {
            float f = fx_feature(seed, dist, (uint64_t)v, (uint64_t)j);
            int64_t o = (v - v0) * d + j;
            if (out_dtype == 0) ((float*)out)[o] = f;
            else if (out_dtype == 1) ((uint16_t*)out)[o] = fx_f32_to_bf16(f);
            else ((uint16_t*)out)[o] = fx_f32_to_f16(f);
        }
    }
}

/*
 * The same rows as fx_features, as a chunk-loader fill callback: ctx is an
 * fx_fill_ctx, rows [v0, v1) go to out.  The row's hash prefix
 * H(seed, 2, v) is taken once per row (the values are fx_features' exactly);
 * rows are spread over ctx->threads OpenMP threads (0: the runtime's
 * default).  Returns 0.
 */
typedef struct {
    uint64_t seed;
    int32_t dist;
    int32_t out_dtype;
    int64_t d;
    int32_t threads;
} fx_fill_ctx;

int fx_fill_features(void* ctx_, int64_t v0, int64_t v1, void* out) {
    const fx_fill_ctx* ctx = (const fx_fill_ctx*)ctx_;
    const uint64_t s2 = fx_step(ctx->seed, 2);
    const int64_t d = ctx->d;
    const int nt = ctx->threads > 0 ? ctx->threads : omp_get_max_threads();
#pragma omp parallel for schedule(static) num_threads(nt)
    for (int64_t v = v0; v < v1; v++) {
        const uint64_t hv = fx_step(s2, (uint64_t)v);
        const int64_t o = (v - v0) * d;
        if (ctx->dist == 0 && ctx->out_dtype == 0) {
            fx_uniform_row(hv, d, (float*)out + o);
            continue;
        }
        for (int64_t j = 0; j < d; j++) {
            float f = fx_feature(ctx->seed, ctx->dist, (uint64_t)v, (uint64_t)j);
            if (ctx->out_dtype == 0) ((float*)out)[o + j] = f;
            else if (ctx->out_dtype == 1) ((uint16_t*)out)[o + j] = fx_f32_to_bf16(f);
            else ((uint16_t*)out)[o + j] = fx_f32_to_f16(f);
        }
    }
    return 0;
}

/* Rows listed in `ids` (any order), for sampled checks at large sizes. */
void fx_features_rows(uint64_t seed, int dist, int64_t nids, const int64_t* ids, int64_t d, int out_dtype, void* out) {
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < nids; r++) {
        for (int64_t j = 0; j < d; j++) {
            float f = fx_feature(seed, dist, (uint64_t)ids[r], (uint64_t)j);
            int64_t o = r * d + j;
            if (out_dtype == 0) ((float*)out)[o] = f;
            else if (out_dtype == 1) ((uint16_t*)out)[o] = fx_f32_to_bf16(f);
            else ((uint16_t*)out)[o] = fx_f32_to_f16(f);
        }
    }
}

/* ------------------------------------------------------ weights / bias ---- */
/*
 * Xavier-uniform (Glorot and Bengio, 2010), gain 1: a = sqrt(6/(fan_in+fan_out)),
 * entry (i, j) = a * (2 * ((H(seed,3,layer,i,j) >> 40) * 2^-24) - 1), in fp64,
 * rounded to fp32.  The matrix is the one that maps an input vector to an
 * output vector, rows = output width, cols = input width (for the
 * concatenated GraphSAGE update, cols = 2 * input width).
 */
void fx_weights(uint64_t seed, int64_t layer, int64_t rows, int64_t cols,
                int64_t fan_in, int64_t fan_out, float* out) {
    double a = sqrt(6.0 / (double)(fan_in + fan_out));
    for (int64_t i = 0; i < rows; i++)
        for (int64_t j = 0; j < cols; j++) {
            uint64_t h = fx_step(fx_step(fx_step(fx_step(seed, 3), (uint64_t)layer), (uint64_t)i), (uint64_t)j);
            double u = (double)(h >> 40) * 0x1.0p-24;
            out[i * cols + j] = (float)(a * (2.0 * u - 1.0));
        }
}

/* bias_j = (1/sqrt(fan_in)) * (2 * ((H(seed,6,layer,j) >> 40) * 2^-24) - 1), fp32 */
void fx_bias(uint64_t seed, int64_t layer, int64_t d, int64_t fan_in, float* out) {
    double bound = 1.0 / sqrt((double)fan_in);
    for (int64_t j = 0; j < d; j++) {
        uint64_t h = fx_step(fx_step(fx_step(seed, 6), (uint64_t)layer), (uint64_t)j);
        double u = (double)(h >> 40) * 0x1.0p-24;
        out[j] = (float)(bound * (2.0 * u - 1.0));
    }
}

/* Attention vectors of a GAT layer, a (2 x d) matrix: row 0 multiplies the
 * transformed source row, row 1 the transformed destination row;
 * a_kj = sqrt(6 / (d + 1)) * (2 * ((H(seed,8,layer,k,j) >> 40) * 2^-24) - 1), fp32 */
void fx_attention(uint64_t seed, int64_t layer, int64_t d, float* out) {
    double a = sqrt(6.0 / (double)(d + 1));
    for (int64_t k = 0; k < 2; k++)
        for (int64_t j = 0; j < d; j++) {
            uint64_t h = fx_step(fx_step(fx_step(fx_step(seed, 8), (uint64_t)layer), (uint64_t)k), (uint64_t)j);
            double u = (double)(h >> 40) * 0x1.0p-24;
            out[k * d + j] = (float)(a * (2.0 * u - 1.0));
        }
}

/* Round an fp32 array to bf16 (dtype 1) or fp16 (dtype 2), RNE. */
void fx_round16(int64_t n, const float* in, int dtype, uint16_t* out) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++) out[i] = dtype == 1 ? fx_f32_to_bf16(in[i]) : fx_f32_to_f16(in[i]);
}

/* ------------------------------------------------------ random vertex IDs - */
/* new_id(v) = rank of (H(seed,5,v,0), v) in ascending order. */
typedef struct { uint64_t k; int64_t v; } fx_kv;
static int fx_kv_cmp(const void* a, const void* b) {
    const fx_kv* x = (const fx_kv*)a; const fx_kv* y = (const fx_kv*)b;
    if (x->k != y->k) return x->k < y->k ? -1 : 1;
    return (x->v > y->v) - (x->v < y->v);
}
int fx_random_ids(uint64_t seed, int64_t n, int32_t* new_of_old) {
    fx_kv* a = (fx_kv*)malloc((size_t)n * sizeof(fx_kv));
    if (!a) return -2;
#pragma omp parallel for schedule(static)
    for (int64_t v = 0; v < n; v++) {
        a[v].k = fx_step(fx_step(fx_step(seed, 5), (uint64_t)v), 0);
        a[v].v = v;
    }
    qsort(a, (size_t)n, sizeof(fx_kv), fx_kv_cmp);
    for (int64_t r = 0; r < n; r++) new_of_old[a[r].v] = (int32_t)r;
    free(a);
    return 0;
}

/* Apply a vertex relabelling to an edge list in place. */
void fx_relabel_edges(int64_t e, const int32_t* new_of_old, int32_t* src, int32_t* dst) {
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < e; i++) { src[i] = new_of_old[src[i]]; dst[i] = new_of_old[dst[i]]; }
}
