// One GNN layer as source-centric broadcast (Taurus, Sec. 3.1-3.6).
//
// Per layer (taurus_layer_init):
//   - pending[v] = |M(v)| + 1: every propagated in-edge and the vertex's own
//     self message each count as one arrival (Sec. 3.4: O(|V|) pending
//     counts; a vertex completes when its count reaches zero);
//   - the chunk index: all propagated in-edges (u, v) plus one self item
//     (v, v) per vertex, stably sorted by (chunk of the source, v).  In
//     chunk j the messages to one destination are then one contiguous
//     segment, with sources ascending and the self item last;
//   - the segments that straddle scatter tiles, so their partial sums can be
//     combined in a fixed order after the tile pass (no float atomics).
// Per chunk (taurus_push_chunk):
//   1. transform: Y = X_c W (GCN rows scaled by d^_out(u)^-1/2; GraphSAGE
//      Y = [X_c W_agg^T | X_c W_self^T]);
//   2. scatter: for every segment, the sum of its source rows scaled once by
//      1/|M(v)| (the per-message normalisation of Sec. 3.4 applied to the
//      segment sum) plus the self row, added to v's fp32 accumulator; the
//      pending count drops by the segment length;
//   3. finalise in place: the flush that brings pending[v] to zero writes
//      out[v] = act(phi_v * acc[v] + b) directly (GCN phi_v = d^_in(v)^-1/2,
//      GraphSAGE phi_v = 1), the graduation step of Sec. 3.6;
//   4. fix-up: segments cut by tile boundaries are summed from per-tile
//      carries and flushed the same way.
// A flush is the only writer of its destination within a kernel (segments
// of one chunk are disjoint, kernels of one layer are stream ordered), so
// accumulators are updated with plain loads and stores.
#include <algorithm>
#include <chrono>

#include "internal.hpp"

namespace taurus {

int build_csr_impl(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                   int32_t* col_dst, hipStream_t s);
void gemm_f32(const float* X, int64_t M, int K, const float* Wp, int Nc, const float* rscale, float* Y,
              hipStream_t s);
void gemm_pack_weights_f32(const float* W, int K, int Nc, std::vector<float>& packed);
const char* last_error_cstr();

constexpr uint32_t SELF_BIT = 0x80000000u;
constexpr int SC_THREADS = 256;
constexpr int SC_TILE = 1024;

// ------------------------------------------------------------ init kernels --

__global__ void k_in_degree(const int32_t* __restrict__ col_dst, int64_t e, int32_t* __restrict__ deg_in) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < e) atomicAdd(&deg_in[col_dst[i]], 1);
}

// pending and expected arrival counts: |M(v)| propagated messages + 1 self
__global__ void k_init_counts(const int32_t* __restrict__ m, int64_t n, int2* __restrict__ cnt) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n) {
        const int x = m[v] + 1;
        cnt[v] = make_int2(x, x);
    }
}

// GCN source factor d^_out(u)^-1/2 with d^_out = out-degree + 1
__global__ void k_out_norm(const int64_t* __restrict__ row_off, int64_t n, float* __restrict__ n_out) {
    const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (u < n) n_out[u] = 1.0f / sqrtf((float)(row_off[u + 1] - row_off[u] + 1));
}

// Caller-supplied CSR: row_off[0] = 0, row_off[n] = e, non-decreasing, and
// every col_dst in [0, n).  Checked before any kernel indexes with them.
__global__ void k_validate_graph(const int64_t* __restrict__ row_off, const int32_t* __restrict__ col_dst,
                                 int64_t n, int64_t e, int* __restrict__ bad) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0 && (row_off[0] != 0 || row_off[n] != e)) atomicOr(bad, 1);
    if (i < n && row_off[i] > row_off[i + 1]) atomicOr(bad, 1);
    if (i < e) {
        const int32_t c = col_dst[i];
        if (c < 0 || (int64_t)c >= n) atomicOr(bad, 2);
    }
}

// Chunk-index items.  CSR edge i (source u = the row containing i) becomes
// key (chunk(u) << vbits | v), value u - chunk(u)*C; a dropped edge gets
// chunk = nchunks so it sorts after every kept item.  Vertex v's self item
// is (chunk(v) << vbits | v, (v - chunk(v)*C) | SELF_BIT).
__global__ void k_make_items(const int64_t* __restrict__ row_off, const int32_t* __restrict__ col_dst,
                             int64_t e, int64_t n, int64_t C, int64_t nchunks, int vbits,
                             const uint64_t* __restrict__ mask, uint64_t* __restrict__ keys,
                             uint32_t* __restrict__ vals, int* __restrict__ bad) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < e) {
        int64_t lo = 0, hi = n;  // largest u with row_off[u] <= i
        while (hi - lo > 1) {
            const int64_t mid = (lo + hi) >> 1;
            if (row_off[mid] <= i) lo = mid;
            else hi = mid;
        }
        const int64_t u = lo, v = col_dst[i];
        // rows strictly ascending, no self loops (a simple graph)
        if (v == u || (i > row_off[u] && col_dst[i - 1] >= v)) atomicOr(bad, 4);
        const bool kept = !mask || ((mask[i >> 6] >> (i & 63)) & 1ull);
        const int64_t ch = kept ? u / C : nchunks;
        keys[i] = ((uint64_t)ch << vbits) | (uint64_t)v;
        vals[i] = (uint32_t)(u - (u / C) * C);
    } else if (i < e + n) {
        const int64_t v = i - e, ch = v / C;
        keys[i] = ((uint64_t)ch << vbits) | (uint64_t)v;
        vals[i] = (uint32_t)(v - ch * C) | SELF_BIT;
    }
}

// offs[j] = first sorted position whose chunk field is >= j, j in [0, nchunks]
__global__ void k_chunk_bounds(const uint64_t* __restrict__ keys, int64_t total, int64_t nchunks, int vbits,
                               int64_t* __restrict__ offs) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j > nchunks) return;
    const uint64_t target = (uint64_t)j << vbits;
    int64_t lo = 0, hi = total;
    while (lo < hi) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (keys[mid] < target) lo = mid + 1;
        else hi = mid;
    }
    offs[j] = lo;
}

// number of distinct (chunk, destination) pairs among the first `total` keys
__global__ void k_count_pairs(const uint64_t* __restrict__ keys, int64_t total,
                              unsigned long long* __restrict__ pairs) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool head = i < total && (i == 0 || keys[i] != keys[i - 1]);
    const uint64_t b = __ballot(head);
    if ((threadIdx.x & 63) == 0 && b) atomicAdd(pairs, (unsigned long long)__popcll(b));
}

__global__ void k_split_items(const uint64_t* __restrict__ keys, const uint32_t* __restrict__ vals,
                              int64_t total, int vbits, int32_t* __restrict__ dst, uint32_t* __restrict__ src) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < total) {
        dst[i] = (int32_t)(keys[i] & (((uint64_t)1 << vbits) - 1));
        src[i] = vals[i];
    }
}

__global__ void k_gather_bounds(const int32_t* __restrict__ dst, const int64_t* __restrict__ pos, int64_t np,
                                int2* __restrict__ out) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j < np) out[j] = make_int2(dst[pos[j] - 1], dst[pos[j]]);
}

__global__ void k_count_pending(const int2* __restrict__ cnt, int64_t n, unsigned long long* __restrict__ left) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const bool open = v < n && cnt[v].x != 0;
    const uint64_t b = __ballot(open);
    if ((threadIdx.x & 63) == 0 && b) atomicAdd(left, (unsigned long long)__popcll(b));
}

// ---------------------------------------------------------- scatter kernels --

struct ScatterParams {
    const float* Y;        // chunk transform, row stride ystride floats
    int64_t ystride;
    int self_col;          // column offset of the self half (GraphSAGE) or 0 (GCN)
    const int32_t* dst;    // chunk items: destination
    const uint32_t* src;   // chunk items: local source row | SELF_BIT
    int64_t nitems;
    int2* cnt;             // {pending, expected}
    float* acc;            // [n][d_o] fp32 accumulators
    int d_o;
    int agg;               // 0 GraphSAGE-mean, 1 GCN
    int relu;
    int out_dtype;         // 0 fp32, 1 bf16, 2 fp16
    const float* bias;     // [d_o]
    void* out;             // [n][d_o]
    float* carry;          // per tile: [2][d_o] partial contributions (left, right piece)
    int32_t* carry_cnt;    // per tile: [2] message counts of the pieces
};

__device__ inline float4 f4_zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
__device__ inline float4 f4_add(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
__device__ inline float4 f4_axpy(float s, float4 a, float4 b) {
    return make_float4(fmaf(s, a.x, b.x), fmaf(s, a.y, b.y), fmaf(s, a.z, b.z), fmaf(s, a.w, b.w));
}

__device__ inline uint32_t f32_to_bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
__device__ inline uint32_t f32_to_f16_bits(float f) {
    const _Float16 h = (_Float16)f;  // v_cvt_f16_f32, round to nearest even
    return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

__device__ inline void store_out4(void* out, int dtype, int64_t idx, float4 z) {
    if (dtype == 0) {
        *reinterpret_cast<float4*>(static_cast<float*>(out) + idx) = z;
    } else {
        uint2 p;
        if (dtype == 1) {
            p.x = f32_to_bf16_bits(z.x) | (f32_to_bf16_bits(z.y) << 16);
            p.y = f32_to_bf16_bits(z.z) | (f32_to_bf16_bits(z.w) << 16);
        } else {
            p.x = f32_to_f16_bits(z.x) | (f32_to_f16_bits(z.y) << 16);
            p.y = f32_to_f16_bits(z.z) | (f32_to_f16_bits(z.w) << 16);
        }
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(out) + idx) = p;
    }
}

__device__ inline float seg_scale(int agg, int expect) {
    // GraphSAGE-mean: 1/|M(v)| (|M(v)| = expect - 1); GCN: sources are pre-scaled
    return agg == 0 ? (expect > 1 ? 1.0f / (float)(expect - 1) : 0.0f) : 1.0f;
}

// Sole-owner flush of contribution c (already scaled) carrying `count`
// messages to v.  pe = {pending, expected} as read before the flush.
template <int G, int VEC>
__device__ inline void flush_owner(const ScatterParams& p, int v, int2 pe, const float4 (&c)[VEC], int count,
                                   int lane) {
    const int left = pe.x - count;
    const bool fresh = pe.x == pe.y;  // nothing accumulated yet: acc[v] is logically zero
    float* arow = p.acc + (int64_t)v * p.d_o;
    if (left == 0) {
        const float phi = p.agg == 1 ? 1.0f / sqrtf((float)pe.y) : 1.0f;
#pragma unroll
        for (int j = 0; j < VEC; j++) {
            const int col = (j * G + lane) * 4;
            if (col < p.d_o) {
                float4 t = fresh ? c[j] : f4_add(*reinterpret_cast<const float4*>(arow + col), c[j]);
                const float4 b = *reinterpret_cast<const float4*>(p.bias + col);
                float4 z = f4_axpy(phi, t, b);
                if (p.relu) {
                    z.x = fmaxf(z.x, 0.f); z.y = fmaxf(z.y, 0.f);
                    z.z = fmaxf(z.z, 0.f); z.w = fmaxf(z.w, 0.f);
                }
                store_out4(p.out, p.out_dtype, (int64_t)v * p.d_o + col, z);
            }
        }
    } else {
#pragma unroll
        for (int j = 0; j < VEC; j++) {
            const int col = (j * G + lane) * 4;
            if (col < p.d_o) {
                float4 t = fresh ? c[j] : f4_add(*reinterpret_cast<const float4*>(arow + col), c[j]);
                *reinterpret_cast<float4*>(arow + col) = t;
            }
        }
    }
    if (lane == 0) p.cnt[v].x = left;
}

// One workgroup reduces SC_TILE consecutive items of a chunk.  Row-group rg
// (G lanes, one float4 per lane and VEC) walks its own sub-range; runs whose
// segment is entirely inside the sub-range are flushed at once, runs open to
// the left or right are parked in LDS, merged across row-groups, and either
// flushed (closed inside the tile) or left as the tile's carry.
template <int G, int VEC>
__global__ __launch_bounds__(SC_THREADS) void k_scatter(ScatterParams p) {
    constexpr int NRG = SC_THREADS / G;
    constexpr int PER = SC_TILE / NRG;
    __shared__ int32_t s_dst[SC_TILE];
    __shared__ uint32_t s_src[SC_TILE];
    __shared__ int s_pv[2 * NRG], s_pc[2 * NRG], s_pf[2 * NRG];
    __shared__ float4 s_prow[2 * NRG][G * VEC];

    const int tid = threadIdx.x, rg = tid / G, lane = tid % G;
    const int64_t t0 = (int64_t)blockIdx.x * SC_TILE;
    const int nt = (int)min((int64_t)SC_TILE, p.nitems - t0);
    for (int i = tid; i < nt; i += SC_THREADS) {
        s_dst[i] = p.dst[t0 + i];
        s_src[i] = p.src[t0 + i];
    }
    if (tid < 2 * NRG) {
        s_pv[tid] = -1;
        s_pc[tid] = 0;
        s_pf[tid] = 0;
    }
    const int prev_v = t0 > 0 ? p.dst[t0 - 1] : -1;
    const int next_v = t0 + nt < p.nitems ? p.dst[t0 + nt] : -1;
    __syncthreads();

    const int a = rg * PER, b = min(a + PER, nt);
    if (a < b) {
        const bool lopen = (a > 0 ? s_dst[a - 1] : prev_v) == s_dst[a];
        int cur = s_dst[a], count = 0;
        bool first = true;
        float4 sa[VEC], ss[VEC];
#pragma unroll
        for (int j = 0; j < VEC; j++) sa[j] = ss[j] = f4_zero();
        auto emit = [&](bool lo, bool ro) {
            const int2 pe = p.cnt[cur];
            const float sig = seg_scale(p.agg, pe.y);
            float4 c[VEC];
#pragma unroll
            for (int j = 0; j < VEC; j++) c[j] = f4_axpy(sig, sa[j], ss[j]);
            if (!lo && !ro) {
                flush_owner<G, VEC>(p, cur, pe, c, count, lane);
            } else {
                const int slot = 2 * rg + (lo ? 0 : 1);
#pragma unroll
                for (int j = 0; j < VEC; j++) s_prow[slot][j * G + lane] = c[j];
                if (lane == 0) {
                    s_pv[slot] = cur;
                    s_pc[slot] = count;
                    s_pf[slot] = (lo ? 1 : 0) | (ro ? 2 : 0);
                }
            }
        };
        for (int i = a; i < b; i++) {
            const int v = s_dst[i];
            if (v != cur) {
                emit(first && lopen, false);
                first = false;
                cur = v;
                count = 0;
#pragma unroll
                for (int j = 0; j < VEC; j++) sa[j] = ss[j] = f4_zero();
            }
            const uint32_t code = s_src[i];
            const bool self = (code & SELF_BIT) != 0;
            const float* row = p.Y + (int64_t)(code & ~SELF_BIT) * p.ystride + (self ? p.self_col : 0);
#pragma unroll
            for (int j = 0; j < VEC; j++) {
                const int col = (j * G + lane) * 4;
                if (col < p.d_o) {
                    const float4 y = *reinterpret_cast<const float4*>(row + col);
                    if (self) ss[j] = f4_add(ss[j], y);
                    else sa[j] = f4_add(sa[j], y);
                }
            }
            count++;
        }
        const bool ropen = (b < nt ? s_dst[b] : next_v) == cur;
        emit(first && lopen, ropen);
    }
    __syncthreads();

    // merge parked pieces: the row-group owning the first slot of a run of
    // equal destinations sums the run
#pragma unroll
    for (int q = 0; q < 2; q++) {
        const int s = 2 * rg + q;
        const int v = s_pv[s];
        if (v < 0) continue;
        int ps = s - 1;
        while (ps >= 0 && s_pv[ps] < 0) ps--;
        if (ps >= 0 && s_pv[ps] == v) continue;
        float4 c[VEC];
#pragma unroll
        for (int j = 0; j < VEC; j++) c[j] = s_prow[s][j * G + lane];
        int count = s_pc[s], last = s;
        for (int ns = s + 1; ns < 2 * NRG; ns++) {
            const int w = s_pv[ns];
            if (w < 0) continue;
            if (w != v) break;
#pragma unroll
            for (int j = 0; j < VEC; j++) c[j] = f4_add(c[j], s_prow[ns][j * G + lane]);
            count += s_pc[ns];
            last = ns;
        }
        const bool lo = (s_pf[s] & 1) != 0, ro = (s_pf[last] & 2) != 0;
        if (!lo && !ro) {
            flush_owner<G, VEC>(p, v, p.cnt[v], c, count, lane);
        } else {
            const int side = lo ? 0 : 1;
            float* crow = p.carry + ((int64_t)blockIdx.x * 2 + side) * p.d_o;
#pragma unroll
            for (int j = 0; j < VEC; j++) {
                const int col = (j * G + lane) * 4;
                if (col < p.d_o) *reinterpret_cast<float4*>(crow + col) = c[j];
            }
            if (lane == 0) p.carry_cnt[blockIdx.x * 2 + side] = count;
        }
    }
}

// A segment cut by tile boundaries spans tiles t0..t1: its pieces are the
// right carry of t0 and the left carries of t0+1..t1, summed in that order.
template <int G, int VEC>
__global__ __launch_bounds__(SC_THREADS) void k_fixup(ScatterParams p, const int4* __restrict__ fix, int64_t nfix) {
    constexpr int NRG = SC_THREADS / G;
    const int rg = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t idx = (int64_t)blockIdx.x * NRG + rg;
    if (idx >= nfix) return;
    const int4 f = fix[idx];
    const int v = f.x, ta = f.y, tb = f.z;
    float4 c[VEC];
    const float* crow = p.carry + ((int64_t)ta * 2 + 1) * p.d_o;
#pragma unroll
    for (int j = 0; j < VEC; j++) {
        const int col = (j * G + lane) * 4;
        c[j] = col < p.d_o ? *reinterpret_cast<const float4*>(crow + col) : f4_zero();
    }
    int count = p.carry_cnt[ta * 2 + 1];
    for (int t = ta + 1; t <= tb; t++) {
        const float* lrow = p.carry + ((int64_t)t * 2) * p.d_o;
#pragma unroll
        for (int j = 0; j < VEC; j++) {
            const int col = (j * G + lane) * 4;
            if (col < p.d_o) c[j] = f4_add(c[j], *reinterpret_cast<const float4*>(lrow + col));
        }
        count += p.carry_cnt[t * 2];
    }
    flush_owner<G, VEC>(p, v, p.cnt[v], c, count, lane);
}

typedef void (*scatter_fn)(ScatterParams);
typedef void (*fixup_fn)(ScatterParams, const int4*, int64_t);

template <int G, int VEC>
static void launch_scatter(const ScatterParams& p, int64_t ntiles, hipStream_t s) {
    k_scatter<G, VEC><<<(unsigned)ntiles, SC_THREADS, 0, s>>>(p);
}
template <int G, int VEC>
static void launch_fixup(const ScatterParams& p, const int4* fix, int64_t nfix, hipStream_t s) {
    constexpr int NRG = SC_THREADS / G;
    k_fixup<G, VEC><<<(unsigned)ceil_div(nfix, NRG), SC_THREADS, 0, s>>>(p, fix, nfix);
}

// lanes per row-group: one float4 per lane up to 64 lanes, then VEC float4s
static void row_group_shape(int d_o, int* G, int* VEC) {
    const int q = (d_o + 3) / 4;
    int g = 4;
    while (g < q && g < 64) g <<= 1;
    int vec = (q + g - 1) / g;
    if (vec == 3) vec = 4;
    *G = g;
    *VEC = vec;
}

static void dispatch_scatter(int G, int VEC, const ScatterParams& p, int64_t ntiles, hipStream_t s) {
    switch (G * 10 + VEC) {
        case 41: launch_scatter<4, 1>(p, ntiles, s); break;
        case 81: launch_scatter<8, 1>(p, ntiles, s); break;
        case 161: launch_scatter<16, 1>(p, ntiles, s); break;
        case 321: launch_scatter<32, 1>(p, ntiles, s); break;
        case 641: launch_scatter<64, 1>(p, ntiles, s); break;
        case 642: launch_scatter<64, 2>(p, ntiles, s); break;
        case 644: launch_scatter<64, 4>(p, ntiles, s); break;
        default: fail(TAURUS_E_INVALID, "unsupported row shape G=%d VEC=%d", G, VEC);
    }
    TAURUS_CHECK_LAUNCH();
}
static void dispatch_fixup(int G, int VEC, const ScatterParams& p, const int4* fix, int64_t nfix, hipStream_t s) {
    switch (G * 10 + VEC) {
        case 41: launch_fixup<4, 1>(p, fix, nfix, s); break;
        case 81: launch_fixup<8, 1>(p, fix, nfix, s); break;
        case 161: launch_fixup<16, 1>(p, fix, nfix, s); break;
        case 321: launch_fixup<32, 1>(p, fix, nfix, s); break;
        case 641: launch_fixup<64, 1>(p, fix, nfix, s); break;
        case 642: launch_fixup<64, 2>(p, fix, nfix, s); break;
        case 644: launch_fixup<64, 4>(p, fix, nfix, s); break;
        default: fail(TAURUS_E_INVALID, "unsupported row shape G=%d VEC=%d", G, VEC);
    }
    TAURUS_CHECK_LAUNCH();
}

}  // namespace taurus

// ------------------------------------------------------------- layer state --

struct taurus_layer {
    taurus_graph g{};
    taurus_layer_desc d{};
    hipStream_t s = nullptr;
    taurus::Arena arena;
    bool poisoned = false;
    int64_t n = 0, C = 0, nchunks = 0, messages = 0, pairs = 0, ntiles_total = 0;
    int d_o = 0, ncols = 0, G = 0, VEC = 0, max_tiles = 0;
    int2* cnt = nullptr;
    float* n_out = nullptr;
    float* acc = nullptr;
    float* wpack = nullptr;
    float* bias = nullptr;
    float* Y = nullptr;
    int32_t* item_dst = nullptr;
    uint32_t* item_src = nullptr;
    int4* fix = nullptr;
    float* carry = nullptr;
    int32_t* carry_cnt = nullptr;
    uint64_t* mask = nullptr;
    std::vector<int64_t> chunk_off, fix_off;
    std::vector<uint8_t> pushed;
    int64_t npushed = 0;
    double ms_init = 0;
    std::vector<hipEvent_t> events;  // 4 per pushed chunk when profiling
    ~taurus_layer() {
        for (auto ev : events) (void)hipEventDestroy(ev);
    }
};

namespace taurus {

static void validate(const taurus_graph* g, const taurus_layer_desc* d) {
    if (!g || !d) fail(TAURUS_E_INVALID, "null graph or descriptor");
    if (g->n <= 0 || g->n >= ((int64_t)1 << 31) || g->e < 0)
        fail(TAURUS_E_INVALID, "graph size n=%lld e=%lld out of range", (long long)g->n, (long long)g->e);
    if (!g->row_off || (g->e > 0 && !g->col_dst)) fail(TAURUS_E_INVALID, "graph arrays are null");
    if (d->agg != TAURUS_SAGE_MEAN && d->agg != TAURUS_GCN_SYM) fail(TAURUS_E_INVALID, "unknown agg %d", d->agg);
    if (d->d_in <= 0 || d->d_out <= 0 || d->d_in % 4 || d->d_out % 4 || d->d_out > 1024 || d->d_in > 8192)
        fail(TAURUS_E_INVALID, "d_in=%d d_out=%d: widths must be positive multiples of 4, d_out <= 1024",
             d->d_in, d->d_out);
    if (d->in_dtype != TAURUS_F32)
        fail(TAURUS_E_INVALID, "in_dtype %d: only fp32 layer inputs are supported by this build", d->in_dtype);
    if (d->out_dtype < 0 || d->out_dtype > 2) fail(TAURUS_E_INVALID, "out_dtype %d", d->out_dtype);
    if (!d->weight) fail(TAURUS_E_INVALID, "weight is null");
    if (d->chunk <= 0 || d->chunk >= ((int64_t)1 << 31)) fail(TAURUS_E_INVALID, "chunk %lld", (long long)d->chunk);
    if (d->fanout < 0) fail(TAURUS_E_INVALID, "fanout %d", d->fanout);
    if (d->fanout > 0) fail(TAURUS_E_INVALID, "fanout sampling is not supported by this build");
    if (d->agg == TAURUS_GCN_SYM && d->fanout > 0) fail(TAURUS_E_INVALID, "GCN is defined for exact inference only");
    if (!d->out) fail(TAURUS_E_INVALID, "out is null");
    if (d->out_on_host != 0) fail(TAURUS_E_INVALID, "out_on_host=%d is not supported by this build", d->out_on_host);
    if (d->hbm_budget < 0) fail(TAURUS_E_INVALID, "hbm_budget < 0");
}

static void layer_init(taurus_layer* L) {
    const auto t_start = std::chrono::steady_clock::now();
    hipStream_t s = L->s;
    const taurus_graph& g = L->g;
    const taurus_layer_desc& d = L->d;
    const int64_t n = g.n, e = g.e, C = d.chunk;
    L->n = n;
    L->C = C;
    L->nchunks = ceil_div(n, C);
    L->d_o = d.d_out;
    L->ncols = d.agg == TAURUS_SAGE_MEAN ? 2 * d.d_out : d.d_out;
    row_group_shape(L->d_o, &L->G, &L->VEC);
    const int T = 256;
    Arena tmp;  // init-only temporaries

    // the caller's graph must be a valid simple CSR before anything indexes with it
    int* bad = tmp.alloc<int>(1, "graph flag");
    TAURUS_HIP(hipMemsetAsync(bad, 0, sizeof(int), s));
    k_validate_graph<<<(unsigned)ceil_div(std::max(n, e), T), T, 0, s>>>(g.row_off, g.col_dst, n, e, bad);
    TAURUS_CHECK_LAUNCH();
    int hbad = 0;
    TAURUS_HIP(hipMemcpyAsync(&hbad, bad, sizeof(int), hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    if (hbad) fail(TAURUS_E_INVALID, "graph is not a valid CSR over [0, n) (flags %d)", hbad);

    // degrees and arrival counts
    int32_t* m = tmp.alloc<int32_t>(n, "in-degrees");
    TAURUS_HIP(hipMemsetAsync(m, 0, (size_t)n * 4, s));
    if (e > 0) {
        k_in_degree<<<(unsigned)ceil_div(e, T), T, 0, s>>>(g.col_dst, e, m);
        TAURUS_CHECK_LAUNCH();
    }
    L->messages = e;
    L->cnt = L->arena.alloc<int2>(n, "pending counts");
    k_init_counts<<<(unsigned)ceil_div(n, T), T, 0, s>>>(m, n, L->cnt);
    TAURUS_CHECK_LAUNCH();
    if (d.agg == TAURUS_GCN_SYM) {
        L->n_out = L->arena.alloc<float>(n, "source norms");
        k_out_norm<<<(unsigned)ceil_div(n, T), T, 0, s>>>(g.row_off, n, L->n_out);
        TAURUS_CHECK_LAUNCH();
    }

    // weights and bias
    std::vector<float> packed;
    gemm_pack_weights_f32(d.weight, d.d_in, L->ncols, packed);
    L->wpack = L->arena.alloc<float>((int64_t)packed.size(), "packed weights");
    TAURUS_HIP(hipMemcpyAsync(L->wpack, packed.data(), packed.size() * 4, hipMemcpyHostToDevice, s));
    std::vector<float> hb((size_t)L->d_o, 0.0f);
    if (d.bias) std::copy(d.bias, d.bias + L->d_o, hb.begin());
    L->bias = L->arena.alloc<float>(L->d_o, "bias");
    TAURUS_HIP(hipMemcpyAsync(L->bias, hb.data(), hb.size() * 4, hipMemcpyHostToDevice, s));

    // chunk index
    const int vbits = std::max(1, bits_for(n - 1));
    const int cbits = bits_for(L->nchunks);
    if (vbits + cbits > 64) fail(TAURUS_E_INVALID, "key does not fit 64 bits");
    const int64_t total = e + n;
    uint64_t* keys = tmp.alloc<uint64_t>(total, "index keys");
    uint32_t* vals = tmp.alloc<uint32_t>(total, "index values");
    k_make_items<<<(unsigned)ceil_div(total, T), T, 0, s>>>(g.row_off, g.col_dst, e, n, C, L->nchunks, vbits,
                                                            L->mask, keys, vals, bad);
    TAURUS_CHECK_LAUNCH();
    TAURUS_HIP(hipMemcpyAsync(&hbad, bad, sizeof(int), hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    if (hbad) fail(TAURUS_E_INVALID, "graph rows are not strictly ascending or hold a self loop");
    radix_sort_u64(keys, vals, total, vbits + cbits, tmp, s);
    int64_t* doffs = tmp.alloc<int64_t>(L->nchunks + 1, "chunk offsets");
    k_chunk_bounds<<<(unsigned)ceil_div(L->nchunks + 1, T), T, 0, s>>>(keys, total, L->nchunks, vbits, doffs);
    TAURUS_CHECK_LAUNCH();
    L->chunk_off.resize((size_t)L->nchunks + 1);
    TAURUS_HIP(hipMemcpyAsync(L->chunk_off.data(), doffs, (size_t)(L->nchunks + 1) * 8, hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    const int64_t kept_total = L->chunk_off[(size_t)L->nchunks];
    unsigned long long* dpairs = tmp.alloc<unsigned long long>(1, "pair count");
    TAURUS_HIP(hipMemsetAsync(dpairs, 0, 8, s));
    k_count_pairs<<<(unsigned)ceil_div(kept_total, T), T, 0, s>>>(keys, kept_total, dpairs);
    TAURUS_CHECK_LAUNCH();
    L->item_dst = L->arena.alloc<int32_t>(kept_total, "item destinations");
    L->item_src = L->arena.alloc<uint32_t>(kept_total, "item sources");
    k_split_items<<<(unsigned)ceil_div(kept_total, T), T, 0, s>>>(keys, vals, kept_total, vbits, L->item_dst,
                                                                 L->item_src);
    TAURUS_CHECK_LAUNCH();
    unsigned long long hpairs = 0;
    TAURUS_HIP(hipMemcpyAsync(&hpairs, dpairs, 8, hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    L->pairs = (int64_t)hpairs;
    tmp.free_ptr(vals);
    tmp.free_ptr(keys);

    // tiles and the segments that straddle them
    std::vector<int64_t> bpos;
    for (int64_t k = 0; k < L->nchunks; k++) {
        const int64_t cnt_k = L->chunk_off[k + 1] - L->chunk_off[k];
        const int64_t nt = ceil_div(cnt_k, SC_TILE);
        L->ntiles_total += nt;
        L->max_tiles = (int)std::max<int64_t>(L->max_tiles, nt);
        for (int64_t t = 1; t < nt; t++) bpos.push_back(L->chunk_off[k] + t * SC_TILE);
    }
    std::vector<int2> bval(bpos.size());
    if (!bpos.empty()) {
        int64_t* dpos = tmp.alloc<int64_t>((int64_t)bpos.size(), "tile bounds");
        int2* dval = tmp.alloc<int2>((int64_t)bpos.size(), "tile bound values");
        TAURUS_HIP(hipMemcpyAsync(dpos, bpos.data(), bpos.size() * 8, hipMemcpyHostToDevice, s));
        k_gather_bounds<<<(unsigned)ceil_div((int64_t)bpos.size(), T), T, 0, s>>>(L->item_dst, dpos,
                                                                                 (int64_t)bpos.size(), dval);
        TAURUS_CHECK_LAUNCH();
        TAURUS_HIP(hipMemcpyAsync(bval.data(), dval, bpos.size() * sizeof(int2), hipMemcpyDeviceToHost, s));
        TAURUS_HIP(hipStreamSynchronize(s));
    }
    std::vector<int4> hfix;
    L->fix_off.assign((size_t)L->nchunks + 1, 0);
    size_t bi = 0;
    for (int64_t k = 0; k < L->nchunks; k++) {
        L->fix_off[k] = (int64_t)hfix.size();
        const int64_t nt = ceil_div(L->chunk_off[k + 1] - L->chunk_off[k], SC_TILE);
        bool prev_split = false;
        int prev_v = -1;
        for (int64_t t = 1; t < nt; t++, bi++) {
            const int2 bv = bval[bi];  // (dst before, dst at) tile t's first item
            const bool split = bv.x == bv.y;
            if (split) {
                if (prev_split && prev_v == bv.y) hfix.back().z = (int)t;  // tile t-1 lies inside the segment
                else hfix.push_back(make_int4(bv.y, (int)(t - 1), (int)t, 0));
            }
            prev_split = split;
            prev_v = bv.y;
        }
    }
    L->fix_off[(size_t)L->nchunks] = (int64_t)hfix.size();
    if (!hfix.empty()) {
        L->fix = L->arena.alloc<int4>((int64_t)hfix.size(), "fix-up list");
        TAURUS_HIP(hipMemcpyAsync(L->fix, hfix.data(), hfix.size() * sizeof(int4), hipMemcpyHostToDevice, s));
    }

    // working buffers
    L->acc = L->arena.alloc<float>(n * (int64_t)L->d_o, "accumulators");
    L->Y = L->arena.alloc<float>(std::min<int64_t>(C, n) * (int64_t)L->ncols, "chunk transform");
    L->carry = L->arena.alloc<float>((int64_t)std::max(1, L->max_tiles) * 2 * L->d_o, "tile carries");
    L->carry_cnt = L->arena.alloc<int32_t>((int64_t)std::max(1, L->max_tiles) * 2, "tile carry counts");
    L->pushed.assign((size_t)L->nchunks, 0);
    TAURUS_HIP(hipStreamSynchronize(s));
    tmp.release();
    L->ms_init = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_start).count();
}

static void push_chunk(taurus_layer* L, int64_t b, int64_t e, const void* x, int32_t x_on_host) {
    if (L->poisoned) fail(TAURUS_E_STATE, "layer handle is poisoned by an earlier failure");
    if (b < 0 || e > L->n || b >= e || b % L->C != 0 || e != std::min(b + L->C, L->n))
        fail(TAURUS_E_INVALID, "chunk [%lld, %lld) is not a whole chunk of size %lld",
             (long long)b, (long long)e, (long long)L->C);
    if (!x) fail(TAURUS_E_INVALID, "x is null");
    if (x_on_host != 0) fail(TAURUS_E_INVALID, "host-resident chunks are not supported by this build");
    const int64_t k = b / L->C;
    if (L->pushed[(size_t)k]) fail(TAURUS_E_STATE, "chunk %lld pushed twice", (long long)k);
    hipStream_t s = L->s;
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    if (L->d.profile) {
        for (int i = 0; i < 4; i++) {
            TAURUS_HIP(hipEventCreate(&ev[i]));
            L->events.push_back(ev[i]);
        }
        TAURUS_HIP(hipEventRecord(ev[0], s));
    }
    L->pushed[(size_t)k] = 1;
    L->npushed++;
    const int64_t rows = e - b;
    gemm_f32(static_cast<const float*>(x), rows, L->d.d_in, L->wpack, L->ncols, L->n_out ? L->n_out + b : nullptr,
             L->Y, s);
    if (ev[1]) TAURUS_HIP(hipEventRecord(ev[1], s));
    ScatterParams p;
    p.Y = L->Y;
    p.ystride = L->ncols;
    p.self_col = L->d.agg == TAURUS_SAGE_MEAN ? L->d_o : 0;
    p.dst = L->item_dst + L->chunk_off[(size_t)k];
    p.src = L->item_src + L->chunk_off[(size_t)k];
    p.nitems = L->chunk_off[(size_t)k + 1] - L->chunk_off[(size_t)k];
    p.cnt = L->cnt;
    p.acc = L->acc;
    p.d_o = L->d_o;
    p.agg = L->d.agg;
    p.relu = L->d.relu;
    p.out_dtype = L->d.out_dtype;
    p.bias = L->bias;
    p.out = L->d.out;
    p.carry = L->carry;
    p.carry_cnt = L->carry_cnt;
    const int64_t ntiles = ceil_div(p.nitems, SC_TILE);
    if (ntiles > 0) dispatch_scatter(L->G, L->VEC, p, ntiles, s);
    if (ev[2]) TAURUS_HIP(hipEventRecord(ev[2], s));
    const int64_t nfix = L->fix_off[(size_t)k + 1] - L->fix_off[(size_t)k];
    if (nfix > 0) dispatch_fixup(L->G, L->VEC, p, L->fix + L->fix_off[(size_t)k], nfix, s);
    if (ev[3]) TAURUS_HIP(hipEventRecord(ev[3], s));
}

static int finalize(taurus_layer* L, taurus_stats* st) {
    if (L->poisoned) fail(TAURUS_E_STATE, "layer handle is poisoned by an earlier failure");
    hipStream_t s = L->s;
    Arena tmp;
    unsigned long long* dleft = tmp.alloc<unsigned long long>(1, "pending count");
    TAURUS_HIP(hipMemsetAsync(dleft, 0, 8, s));
    k_count_pending<<<(unsigned)ceil_div(L->n, 256), 256, 0, s>>>(L->cnt, L->n, dleft);
    TAURUS_CHECK_LAUNCH();
    unsigned long long left = 0;
    TAURUS_HIP(hipMemcpyAsync(&left, dleft, 8, hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    if (st) {
        std::memset(st, 0, sizeof(*st));
        st->n = L->n;
        st->e = L->g.e;
        st->messages = L->messages;
        st->self_terms = L->n;
        st->pairs = L->pairs;
        st->pending_left = (int64_t)left;
        st->completed = L->n - (int64_t)left;
        st->chunks = L->nchunks;
        st->chunks_pushed = L->npushed;
        st->tiles = L->ntiles_total;
        st->split_segments = L->fix_off.empty() ? 0 : L->fix_off.back();
        st->device_bytes = L->arena.peak();
        st->ms_init = L->ms_init;
        for (size_t i = 0; i + 3 < L->events.size(); i += 4) {
            float a = 0, b = 0, c = 0;
            TAURUS_HIP(hipEventElapsedTime(&a, L->events[i], L->events[i + 1]));
            TAURUS_HIP(hipEventElapsedTime(&b, L->events[i + 1], L->events[i + 2]));
            TAURUS_HIP(hipEventElapsedTime(&c, L->events[i + 2], L->events[i + 3]));
            st->ms_gemm += a;
            st->ms_scatter += b;
            st->ms_fixup += c;
            st->launches_gemm++;
            st->launches_scatter++;
            st->launches_fixup++;
        }
    }
    return left ? TAURUS_E_INCOMPLETE : TAURUS_OK;
}

}  // namespace taurus

// ------------------------------------------------------------------ C ABI --

using namespace taurus;

#define TAURUS_GUARD(body)                                                 \
    try {                                                                  \
        body;                                                              \
    } catch (const Failure& f_) {                                          \
        return f_.status;                                                  \
    } catch (const std::exception& x_) {                                   \
        set_error("internal error: %s", x_.what());                        \
        return TAURUS_E_DEVICE;                                            \
    } catch (...) {                                                        \
        set_error("internal error");                                       \
        return TAURUS_E_DEVICE;                                            \
    }

extern "C" {

const char* taurus_last_error(void) { return last_error_cstr(); }

uint64_t taurus_hash(uint64_t seed, uint64_t tag, int32_t nargs, const uint64_t* args) {
    auto mix = [](uint64_t z) {
        z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
        z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
        return z ^ (z >> 31);
    };
    uint64_t h = mix(seed + 0x9e3779b97f4a7c15ULL + tag);
    for (int i = 0; i < nargs && i < 8; i++) h = mix(h + 0x9e3779b97f4a7c15ULL + args[i]);
    return h;
}

int taurus_build_csr(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                     int32_t* col_dst, void* stream) {
    TAURUS_GUARD(return build_csr_impl(n, e, src, dst, row_off, col_dst, static_cast<hipStream_t>(stream)));
}

int taurus_layer_init(const taurus_graph* g, const taurus_layer_desc* d, taurus_layer** out) {
    if (!out) {
        set_error("out handle pointer is null");
        return TAURUS_E_INVALID;
    }
    *out = nullptr;
    taurus_layer* L = nullptr;
    try {
        validate(g, d);
        L = new taurus_layer();
        L->g = *g;
        L->d = *d;
        L->s = static_cast<hipStream_t>(d->stream);
        L->arena.set_budget(d->hbm_budget);
        layer_init(L);
        *out = L;
        return TAURUS_OK;
    } catch (const Failure& f) {
        delete L;
        return f.status;
    } catch (const std::exception& x) {
        delete L;
        set_error("internal error: %s", x.what());
        return TAURUS_E_DEVICE;
    }
}

int taurus_push_chunk(taurus_layer* L, int64_t src_begin, int64_t src_end, const void* x, int32_t x_on_host) {
    if (!L) {
        set_error("null layer handle");
        return TAURUS_E_INVALID;
    }
    try {
        push_chunk(L, src_begin, src_end, x, x_on_host);
        return TAURUS_OK;
    } catch (const Failure& f) {
        if (f.status == TAURUS_E_OOM || f.status == TAURUS_E_DEVICE) L->poisoned = true;
        return f.status;
    }
}

int taurus_finalize(taurus_layer* L, taurus_stats* stats) {
    if (!L) {
        set_error("null layer handle");
        return TAURUS_E_INVALID;
    }
    try {
        int rc = finalize(L, stats);
        if (rc == TAURUS_E_INCOMPLETE)
            set_error("%lld destinations still have pending messages",
                      (long long)(stats ? stats->pending_left : -1));
        return rc;
    } catch (const Failure& f) {
        if (f.status == TAURUS_E_OOM || f.status == TAURUS_E_DEVICE) L->poisoned = true;
        return f.status;
    }
}

int taurus_sampled_edges(taurus_layer* L, uint64_t* mask_bits_host, int64_t* n_kept) {
    if (!L || !mask_bits_host) {
        set_error("null argument");
        return TAURUS_E_INVALID;
    }
    TAURUS_GUARD({
        const int64_t words = ceil_div(L->g.e, 64);
        if (L->mask) {
            TAURUS_HIP(hipMemcpyAsync(mask_bits_host, L->mask, (size_t)words * 8, hipMemcpyDeviceToHost, L->s));
            TAURUS_HIP(hipStreamSynchronize(L->s));
        } else {
            for (int64_t w = 0; w < words; w++) mask_bits_host[w] = ~0ull;
            if (L->g.e % 64) mask_bits_host[words - 1] = (1ull << (L->g.e % 64)) - 1;
        }
        if (n_kept) *n_kept = L->messages;
        return TAURUS_OK;
    });
}

void taurus_layer_destroy(taurus_layer* L) {
    if (!L) return;
    (void)hipStreamSynchronize(L->s);
    delete L;
}

}  // extern "C"
