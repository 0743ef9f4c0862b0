// One GNN layer as source-centric broadcast (Taurus, Sec. 3.1-3.6).
//
// Per graph and chunk size (the chunk index, shared by exact layers):
//   - all propagated in-edges (u, v) plus one self item (v, v) per vertex,
//     stably sorted by (chunk of the source, v).  In chunk j the messages to
//     one destination are then one contiguous segment, sources ascending and
//     the self item last;
//   - each vertex's arrival count |M(v)| + 1: every propagated in-edge and
//     the self message count once (Sec. 3.4: O(|V|) pending counts; a vertex
//     completes when its count reaches zero);
//   - degree-bucketed work units: a segment of at most SHORT_LEN messages is
//     one short unit (handled by a row-group of lanes); a longer one is cut
//     into pieces of at most PIECE_LEN messages (each handled by a whole
//     wave); a segment cut into several pieces (a hub) is completed by the
//     fix-up pass, which sums the pieces' partial rows in a fixed order.
// Per chunk (taurus_push_chunk):
//   1. transform: Y = X_c W on the matrix cores (GCN rows scaled by
//      d^_out(u)^-1/2; GraphSAGE Y = [X_c W_agg^T | X_c W_self^T]);
//   2. scatter: per unit, the sum of its source rows scaled once by
//      1/|M(v)| (the per-message normalisation of Sec. 3.4 applied to the
//      segment sum) plus the self row, added to v's fp32 accumulator; the
//      pending count drops by the segment length;
//   3. finalise in place: the flush that brings pending[v] to zero writes
//      out[v] = act(phi_v * acc[v] + b) directly (GCN phi_v = d^_in(v)^-1/2,
//      GraphSAGE phi_v = 1), the graduation step of Sec. 3.6;
//   4. fix-up: hub segments sum their pieces and flush the same way.
// A flush is the only writer of its destination within a kernel (segments
// of one chunk are disjoint, kernels of one layer are stream ordered), so
// accumulators are updated with plain loads and stores, no atomics.
#include <algorithm>
#include <chrono>
#include <memory>

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
constexpr int SHORT_LEN = 8;    // segments up to this many messages: one row-group
constexpr int PIECE_LEN = 512;  // longer segments: pieces of this many messages, one wave each

// ------------------------------------------------------------ init kernels --

// pending and expected arrival counts: the number of index items of v,
// i.e. |M(v)| propagated messages + 1 self message
__global__ void k_init_counts(const int32_t* __restrict__ items, int64_t n, int2* __restrict__ cnt) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n) cnt[v] = make_int2(items[v], items[v]);
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

// head[i] = 1 where a new (chunk, destination) segment starts
__global__ void k_seg_heads(const uint64_t* __restrict__ keys, int64_t total, int32_t* __restrict__ head) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < total) head[i] = (i == 0 || keys[i] != keys[i - 1]) ? 1 : 0;
}

// seg_start[s] = first item of segment s; seg_start[P] = total
__global__ void k_seg_starts(const int32_t* __restrict__ head, const int64_t* __restrict__ seg_id, int64_t total,
                             int64_t* __restrict__ seg_start) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < total && head[i]) seg_start[seg_id[i]] = i;
    if (i == 0) seg_start[seg_id[total]] = total;
}

// Per segment: add its length to the destination's item count, and count the
// work units it becomes (short unit, wave pieces, fix-up entry).
__global__ void k_seg_classify(const uint64_t* __restrict__ keys, const int64_t* __restrict__ seg_start, int64_t P,
                               int vbits, int32_t* __restrict__ items_per_v, int32_t* __restrict__ n_short,
                               int32_t* __restrict__ n_long, int32_t* __restrict__ n_fix) {
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= P) return;
    const int64_t b = seg_start[s], len = seg_start[s + 1] - b;
    const uint64_t v = keys[b] & (((uint64_t)1 << vbits) - 1);
    atomicAdd(&items_per_v[v], (int)len);
    const int pieces = len <= SHORT_LEN ? 0 : (int)((len + PIECE_LEN - 1) / PIECE_LEN);
    n_short[s] = len <= SHORT_LEN ? 1 : 0;
    n_long[s] = pieces;
    n_fix[s] = pieces > 1 ? 1 : 0;
}

// Write the work units.  unit = {first item relative to its chunk, length,
// destination, slot}; slot = global wave-unit index for pieces of a hub
// segment (their partial rows go to the carry buffer), else -1.  fix-up
// entry = {destination, first wave-unit index, number of pieces, 0}.
__global__ void k_seg_emit(const uint64_t* __restrict__ keys, const int64_t* __restrict__ seg_start, int64_t P,
                           int vbits, const int64_t* __restrict__ chunk_off, const int64_t* __restrict__ o_short,
                           const int64_t* __restrict__ o_long, const int64_t* __restrict__ o_fix,
                           int4* __restrict__ u_short, int4* __restrict__ u_long, int4* __restrict__ u_fix) {
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= P) return;
    const int64_t b = seg_start[s], len = seg_start[s + 1] - b;
    const uint64_t key = keys[b];
    const int v = (int)(key & (((uint64_t)1 << vbits) - 1));
    const int64_t rel = b - chunk_off[key >> vbits];
    if (len <= SHORT_LEN) {
        u_short[o_short[s]] = make_int4((int)rel, (int)len, v, -1);
        return;
    }
    const int pieces = (int)((len + PIECE_LEN - 1) / PIECE_LEN);
    const int64_t first = o_long[s];
    for (int q = 0; q < pieces; q++) {
        const int64_t off = (int64_t)q * PIECE_LEN;
        const int plen = (int)min((int64_t)PIECE_LEN, len - off);
        u_long[first + q] = make_int4((int)(rel + off), plen, v, pieces > 1 ? (int)(first + q) : -1);
    }
    if (pieces > 1) u_fix[o_fix[s]] = make_int4(v, (int)first, pieces, 0);
}

__global__ void k_take_src(const uint32_t* __restrict__ vals, int64_t total, uint32_t* __restrict__ src) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < total) src[i] = vals[i];
}

// per-chunk starts of the three unit lists: values of the scans at each
// chunk's first segment (chunk_off[nchunks] = total maps to segment P)
__global__ void k_chunk_unit_bases(const int64_t* __restrict__ chunk_off, int64_t nchunks,
                                   const int64_t* __restrict__ seg_id, const int64_t* __restrict__ o_short,
                                   const int64_t* __restrict__ o_long, const int64_t* __restrict__ o_fix,
                                   int64_t* __restrict__ bases) {
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k > nchunks) return;
    const int64_t s = seg_id[chunk_off[k]];
    bases[k * 3 + 0] = o_short[s];
    bases[k * 3 + 1] = o_long[s];
    bases[k * 3 + 2] = o_fix[s];
}

__global__ __launch_bounds__(256) void k_count_pending(const int2* __restrict__ cnt, int64_t n,
                                                       unsigned long long* __restrict__ left) {
    __shared__ unsigned int blk;
    if (threadIdx.x == 0) blk = 0;
    __syncthreads();
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const uint64_t b = __ballot(v < n && cnt[v].x != 0);
    if ((threadIdx.x & 63) == 0 && b) atomicAdd(&blk, (unsigned int)__popcll(b));
    __syncthreads();
    if (threadIdx.x == 0 && blk) atomicAdd(left, (unsigned long long)blk);
}

// ---------------------------------------------------------- scatter kernels --

struct ScatterParams {
    const float* Y;        // chunk transform, row stride ystride floats
    int64_t ystride;
    int self_col;          // column offset of the self half (GraphSAGE) or 0 (GCN)
    const uint32_t* src;   // chunk items: local source row | SELF_BIT
    int2* cnt;             // {pending, expected}
    float* acc;            // [n][d_o] fp32 accumulators
    int d_o;
    int agg;               // 0 GraphSAGE-mean, 1 GCN
    int relu;
    int out_dtype;         // 0 fp32, 1 bf16, 2 fp16
    const float* bias;     // [d_o]
    void* out;             // [n][d_o]
    float* carry;          // per hub piece of the chunk: [d_o] partial contribution
    int32_t* carry_cnt;    // per hub piece: message count
    int64_t long_base;     // global index of the chunk's first wave unit (carry slot 0)
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

// Add the source rows of items first, first + step, ... (fewer than len) of
// the chunk into sa (neighbour messages) and ss (the self message), with B
// row loads in flight at a time.
template <int G, int VEC, int B>
__device__ inline void gather_rows(const ScatterParams& p, int first, int len, int step, int lane,
                                   float4 (&sa)[VEC], float4 (&ss)[VEC]) {
    for (int i0 = 0; i0 < len; i0 += B * step) {
        float4 rows[B][VEC];
        bool self[B];
#pragma unroll
        for (int u = 0; u < B; u++) {
            const int i = i0 + u * step;
            self[u] = false;
#pragma unroll
            for (int j = 0; j < VEC; j++) rows[u][j] = f4_zero();
            if (i < len) {
                const uint32_t code = p.src[first + i];
                self[u] = (code & SELF_BIT) != 0;
                const float* row = p.Y + (int64_t)(code & ~SELF_BIT) * p.ystride + (self[u] ? p.self_col : 0);
#pragma unroll
                for (int j = 0; j < VEC; j++) {
                    const int col = (j * G + lane) * 4;
                    if (col < p.d_o) rows[u][j] = *reinterpret_cast<const float4*>(row + col);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < B; u++)
#pragma unroll
            for (int j = 0; j < VEC; j++) {
                if (self[u]) ss[j] = f4_add(ss[j], rows[u][j]);
                else sa[j] = f4_add(sa[j], rows[u][j]);
            }
    }
}

// Degree-bucketed scatter of one chunk.  Blocks [0, short_blocks) take short
// units, one per row-group of G lanes (SC_THREADS / G units per block); the
// remaining blocks take wave units, one per wave (4 per block): the wave's
// 64/G row-groups split the piece's items, reduce across row-groups with
// cross-lane shuffles, and row-group 0 flushes (or parks the partial row of
// a hub piece in its carry slot).
template <int G, int VEC>
__global__ __launch_bounds__(SC_THREADS) void k_scatter(ScatterParams p, const int4* __restrict__ u_short,
                                                        int64_t n_short, int64_t short_blocks,
                                                        const int4* __restrict__ u_long, int64_t n_long) {
    constexpr int NRG = SC_THREADS / G;
    constexpr int R = 64 / G;
    constexpr int B = 8 / VEC;
    if ((int64_t)blockIdx.x < short_blocks) {
        const int rg = threadIdx.x / G, lane = threadIdx.x % G;
        const int64_t ui = (int64_t)blockIdx.x * NRG + rg;
        if (ui >= n_short) return;
        const int4 w = u_short[ui];
        const int2 pe = p.cnt[w.z];
        float4 sa[VEC], ss[VEC];
#pragma unroll
        for (int j = 0; j < VEC; j++) sa[j] = ss[j] = f4_zero();
        gather_rows<G, VEC, B>(p, w.x, w.y, 1, lane, sa, ss);
        const float sig = seg_scale(p.agg, pe.y);
        float4 c[VEC];
#pragma unroll
        for (int j = 0; j < VEC; j++) c[j] = f4_axpy(sig, sa[j], ss[j]);
        flush_owner<G, VEC>(p, w.z, pe, c, w.y, lane);
        return;
    }
    const int wave = threadIdx.x >> 6, l64 = threadIdx.x & 63;
    const int rg = l64 / G, lane = l64 % G;
    const int64_t ui = ((int64_t)blockIdx.x - short_blocks) * (SC_THREADS / 64) + wave;
    if (ui >= n_long) return;
    const int4 w = u_long[ui];
    const int2 pe = p.cnt[w.z];
    float4 sa[VEC], ss[VEC];
#pragma unroll
    for (int j = 0; j < VEC; j++) sa[j] = ss[j] = f4_zero();
    gather_rows<G, VEC, B>(p, w.x + rg, w.y - rg, R, lane, sa, ss);
#pragma unroll
    for (int d = G; d < 64; d <<= 1)
#pragma unroll
        for (int j = 0; j < VEC; j++) {
            sa[j].x += __shfl_xor(sa[j].x, d, 64); sa[j].y += __shfl_xor(sa[j].y, d, 64);
            sa[j].z += __shfl_xor(sa[j].z, d, 64); sa[j].w += __shfl_xor(sa[j].w, d, 64);
            ss[j].x += __shfl_xor(ss[j].x, d, 64); ss[j].y += __shfl_xor(ss[j].y, d, 64);
            ss[j].z += __shfl_xor(ss[j].z, d, 64); ss[j].w += __shfl_xor(ss[j].w, d, 64);
        }
    if (rg != 0) return;
    const float sig = seg_scale(p.agg, pe.y);
    float4 c[VEC];
#pragma unroll
    for (int j = 0; j < VEC; j++) c[j] = f4_axpy(sig, sa[j], ss[j]);
    if (w.w < 0) {
        flush_owner<G, VEC>(p, w.z, pe, c, w.y, lane);
    } else {
        const int64_t slot = (int64_t)w.w - p.long_base;
        float* crow = p.carry + slot * p.d_o;
#pragma unroll
        for (int j = 0; j < VEC; j++) {
            const int col = (j * G + lane) * 4;
            if (col < p.d_o) *reinterpret_cast<float4*>(crow + col) = c[j];
        }
        if (lane == 0) p.carry_cnt[slot] = w.y;
    }
}

// A hub segment's pieces occupy consecutive carry slots; their partial rows
// are summed in slot order and flushed.
template <int G, int VEC>
__global__ __launch_bounds__(SC_THREADS) void k_fixup(ScatterParams p, const int4* __restrict__ fix, int64_t nfix) {
    constexpr int NRG = SC_THREADS / G;
    const int rg = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t idx = (int64_t)blockIdx.x * NRG + rg;
    if (idx >= nfix) return;
    const int4 f = fix[idx];
    const int v = f.x;
    const int64_t first = (int64_t)f.y - p.long_base;
    float4 c[VEC];
#pragma unroll
    for (int j = 0; j < VEC; j++) c[j] = f4_zero();
    int count = 0;
    for (int q = 0; q < f.z; q++) {
        const float* crow = p.carry + (first + q) * p.d_o;
#pragma unroll
        for (int j = 0; j < VEC; j++) {
            const int col = (j * G + lane) * 4;
            if (col < p.d_o) c[j] = f4_add(c[j], *reinterpret_cast<const float4*>(crow + col));
        }
        count += p.carry_cnt[first + q];
    }
    flush_owner<G, VEC>(p, v, p.cnt[v], c, count, lane);
}

template <int G, int VEC>
static void launch_scatter(const ScatterParams& p, const int4* us, int64_t ns, const int4* ul, int64_t nl,
                           hipStream_t s) {
    constexpr int NRG = SC_THREADS / G;
    const int64_t sb = ceil_div(ns, NRG), lb = ceil_div(nl, SC_THREADS / 64);
    k_scatter<G, VEC><<<(unsigned)(sb + lb), SC_THREADS, 0, s>>>(p, us, ns, sb, ul, nl);
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

#define TAURUS_ROW_SHAPES(X) X(4, 1) X(8, 1) X(16, 1) X(32, 1) X(64, 1) X(64, 2) X(64, 4)

static void dispatch_scatter(int G, int VEC, const ScatterParams& p, const int4* us, int64_t ns, const int4* ul,
                             int64_t nl, hipStream_t s) {
#define TAURUS_CASE(g, v)                              \
    if (G == g && VEC == v) {                          \
        launch_scatter<g, v>(p, us, ns, ul, nl, s);    \
        TAURUS_CHECK_LAUNCH();                         \
        return;                                        \
    }
    TAURUS_ROW_SHAPES(TAURUS_CASE)
#undef TAURUS_CASE
    fail(TAURUS_E_INVALID, "unsupported row shape G=%d VEC=%d", G, VEC);
}
static void dispatch_fixup(int G, int VEC, const ScatterParams& p, const int4* fix, int64_t nfix, hipStream_t s) {
#define TAURUS_CASE(g, v)                              \
    if (G == g && VEC == v) {                          \
        launch_fixup<g, v>(p, fix, nfix, s);           \
        TAURUS_CHECK_LAUNCH();                         \
        return;                                        \
    }
    TAURUS_ROW_SHAPES(TAURUS_CASE)
#undef TAURUS_CASE
    fail(TAURUS_E_INVALID, "unsupported row shape G=%d VEC=%d", G, VEC);
}

}  // namespace taurus


// ------------------------------------------------------------- chunk index --

namespace taurus {

// The structures a layer streams over, fixed by (graph, chunk size, edge
// mask): the item sources grouped by (chunk, destination), per-vertex item
// counts (|M(v)| + 1), and per chunk the short units, the wave units and the
// fix-up entries of hub segments.  Exact layers over one graph and chunk
// size share one index.
struct ChunkIndex {
    Arena arena;
    taurus_graph g{};
    int64_t C = 0, nchunks = 0, kept = 0, pairs = 0;
    int64_t n_short = 0, n_long = 0, n_fix = 0, max_long_per_chunk = 0;
    bool sampled = false;
    int32_t* items_per_v = nullptr;
    uint32_t* item_src = nullptr;
    int4* u_short = nullptr;
    int4* u_long = nullptr;
    int4* u_fix = nullptr;
    std::vector<int64_t> chunk_off, short_off, long_off, fix_off;
    double ms_build = 0;
    ChunkIndex(hipStream_t s, int64_t budget) : arena(s, budget) {}
    // The index may outlive the stream it was built on: wait for the device,
    // then return the memory on the null stream.
    ~ChunkIndex() {
        (void)hipDeviceSynchronize();
        arena.set_stream(nullptr);
        arena.release();
    }
};

static void check_graph_args(const taurus_graph* g) {
    if (!g) fail(TAURUS_E_INVALID, "null graph");
    if (g->n <= 0 || g->n >= ((int64_t)1 << 31) || g->e < 0)
        fail(TAURUS_E_INVALID, "graph size n=%lld e=%lld out of range", (long long)g->n, (long long)g->e);
    if (!g->row_off || (g->e > 0 && !g->col_dst)) fail(TAURUS_E_INVALID, "graph arrays are null");
}

static std::shared_ptr<ChunkIndex> build_index(const taurus_graph& g, int64_t C, const uint64_t* mask,
                                               hipStream_t s, int64_t budget) {
    const auto t_start = std::chrono::steady_clock::now();
    auto idx = std::make_shared<ChunkIndex>(s, budget);
    const int64_t n = g.n, e = g.e;
    idx->g = g;
    idx->C = C;
    idx->nchunks = ceil_div(n, C);
    idx->sampled = mask != nullptr;
    const int T = 256;
    const int64_t nch = idx->nchunks;
    Arena tmp(s);

    // the caller's graph must be a valid simple CSR before anything indexes with it
    int* bad = tmp.alloc<int>(1, "graph flag");
    TAURUS_HIP(hipMemsetAsync(bad, 0, sizeof(int), s));
    k_validate_graph<<<(unsigned)ceil_div(std::max(n, e), T), T, 0, s>>>(g.row_off, g.col_dst, n, e, bad);
    TAURUS_CHECK_LAUNCH();
    int hbad = 0;
    TAURUS_HIP(hipMemcpyAsync(&hbad, bad, sizeof(int), hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    if (hbad) fail(TAURUS_E_INVALID, "graph is not a valid CSR over [0, n) (flags %d)", hbad);

    // items sorted by (source chunk, destination), stably
    const int vbits = std::max(1, bits_for(n - 1));
    const int cbits = bits_for(nch);
    if (vbits + cbits > 64) fail(TAURUS_E_INVALID, "index key does not fit 64 bits");
    const int64_t total = e + n;
    uint64_t* keys = tmp.alloc<uint64_t>(total, "index keys");
    uint32_t* vals = tmp.alloc<uint32_t>(total, "index values");
    k_make_items<<<(unsigned)ceil_div(total, T), T, 0, s>>>(g.row_off, g.col_dst, e, n, C, nch, vbits, mask, keys,
                                                            vals, bad);
    TAURUS_CHECK_LAUNCH();
    TAURUS_HIP(hipMemcpyAsync(&hbad, bad, sizeof(int), hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    if (hbad) fail(TAURUS_E_INVALID, "graph rows are not strictly ascending or hold a self loop");
    radix_sort_u64(keys, vals, total, vbits + cbits, tmp, s);

    int64_t* doffs = tmp.alloc<int64_t>(nch + 1, "chunk offsets");
    k_chunk_bounds<<<(unsigned)ceil_div(nch + 1, T), T, 0, s>>>(keys, total, nch, vbits, doffs);
    TAURUS_CHECK_LAUNCH();
    idx->chunk_off.resize((size_t)nch + 1);
    TAURUS_HIP(hipMemcpyAsync(idx->chunk_off.data(), doffs, (size_t)(nch + 1) * 8, hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    const int64_t kept_total = idx->chunk_off[(size_t)nch];
    idx->kept = kept_total - n;

    // segments: heads, ids, starts
    int32_t* head = tmp.alloc<int32_t>(kept_total, "segment heads");
    int64_t* seg_id = tmp.alloc<int64_t>(kept_total + 1, "segment ids");
    k_seg_heads<<<(unsigned)ceil_div(kept_total, T), T, 0, s>>>(keys, kept_total, head);
    TAURUS_CHECK_LAUNCH();
    scan_i32_to_i64(head, seg_id, kept_total, true, tmp, s);
    int64_t P = 0;
    TAURUS_HIP(hipMemcpyAsync(&P, seg_id + kept_total, 8, hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    idx->pairs = P;
    int64_t* seg_start = tmp.alloc<int64_t>(P + 1, "segment starts");
    k_seg_starts<<<(unsigned)ceil_div(kept_total, T), T, 0, s>>>(head, seg_id, kept_total, seg_start);
    TAURUS_CHECK_LAUNCH();

    // classify segments into work units
    idx->items_per_v = idx->arena.alloc<int32_t>(n, "items per vertex");
    TAURUS_HIP(hipMemsetAsync(idx->items_per_v, 0, (size_t)n * 4, s));
    int32_t* c_short = tmp.alloc<int32_t>(P, "short counts");
    int32_t* c_long = tmp.alloc<int32_t>(P, "wave counts");
    int32_t* c_fix = tmp.alloc<int32_t>(P, "fix counts");
    k_seg_classify<<<(unsigned)ceil_div(P, T), T, 0, s>>>(keys, seg_start, P, vbits, idx->items_per_v, c_short,
                                                          c_long, c_fix);
    TAURUS_CHECK_LAUNCH();
    int64_t* o_short = tmp.alloc<int64_t>(P + 1, "short offsets");
    int64_t* o_long = tmp.alloc<int64_t>(P + 1, "wave offsets");
    int64_t* o_fix = tmp.alloc<int64_t>(P + 1, "fix offsets");
    scan_i32_to_i64(c_short, o_short, P, true, tmp, s);
    scan_i32_to_i64(c_long, o_long, P, true, tmp, s);
    scan_i32_to_i64(c_fix, o_fix, P, true, tmp, s);
    int64_t* dbases = tmp.alloc<int64_t>((nch + 1) * 3, "chunk unit bases");
    k_chunk_unit_bases<<<(unsigned)ceil_div(nch + 1, T), T, 0, s>>>(doffs, nch, seg_id, o_short, o_long, o_fix,
                                                                    dbases);
    TAURUS_CHECK_LAUNCH();
    std::vector<int64_t> bases((size_t)(nch + 1) * 3);
    TAURUS_HIP(hipMemcpyAsync(bases.data(), dbases, bases.size() * 8, hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    idx->short_off.resize((size_t)nch + 1);
    idx->long_off.resize((size_t)nch + 1);
    idx->fix_off.resize((size_t)nch + 1);
    for (int64_t k = 0; k <= nch; k++) {
        idx->short_off[k] = bases[k * 3 + 0];
        idx->long_off[k] = bases[k * 3 + 1];
        idx->fix_off[k] = bases[k * 3 + 2];
    }
    idx->n_short = idx->short_off[nch];
    idx->n_long = idx->long_off[nch];
    idx->n_fix = idx->fix_off[nch];
    for (int64_t k = 0; k < nch; k++)
        idx->max_long_per_chunk = std::max(idx->max_long_per_chunk, idx->long_off[k + 1] - idx->long_off[k]);
    if (idx->n_long >= ((int64_t)1 << 31)) fail(TAURUS_E_INVALID, "too many wave units");
    idx->u_short = idx->arena.alloc<int4>(std::max<int64_t>(1, idx->n_short), "short units");
    idx->u_long = idx->arena.alloc<int4>(std::max<int64_t>(1, idx->n_long), "wave units");
    idx->u_fix = idx->arena.alloc<int4>(std::max<int64_t>(1, idx->n_fix), "fix-up entries");
    k_seg_emit<<<(unsigned)ceil_div(P, T), T, 0, s>>>(keys, seg_start, P, vbits, doffs, o_short, o_long, o_fix,
                                                      idx->u_short, idx->u_long, idx->u_fix);
    TAURUS_CHECK_LAUNCH();
    idx->item_src = idx->arena.alloc<uint32_t>(std::max<int64_t>(1, kept_total), "item sources");
    k_take_src<<<(unsigned)ceil_div(kept_total, T), T, 0, s>>>(vals, kept_total, idx->item_src);
    TAURUS_CHECK_LAUNCH();
    tmp.release();
    TAURUS_HIP(hipStreamSynchronize(s));
    idx->ms_build = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_start).count();
    return idx;
}

}  // namespace taurus

// ------------------------------------------------------------- handles -----

struct taurus_plan {
    taurus_graph g{};
    int64_t chunk = 0;
    std::shared_ptr<taurus::ChunkIndex> idx;
};

struct taurus_layer {
    taurus_graph g{};
    taurus_layer_desc d{};
    hipStream_t s = nullptr;
    taurus::Arena arena;
    std::shared_ptr<taurus::ChunkIndex> idx;
    bool poisoned = false;
    int64_t n = 0, C = 0, nchunks = 0;
    int d_o = 0, ncols = 0, G = 0, VEC = 0;
    int2* cnt = nullptr;
    float* n_out = nullptr;
    float* acc = nullptr;
    float* wpack = nullptr;
    float* bias = nullptr;
    float* Y = nullptr;
    float* carry = nullptr;
    int32_t* carry_cnt = nullptr;
    uint64_t* mask = nullptr;
    std::vector<uint8_t> pushed;
    int64_t npushed = 0;
    double ms_init = 0, ms_index = 0;
    std::vector<hipEvent_t> events;  // 4 per chunk when profiling
    ~taurus_layer() {
        for (auto ev : events)
            if (ev) (void)hipEventDestroy(ev);
    }
};

namespace taurus {

static void validate_desc(const taurus_layer_desc* d) {
    if (!d) fail(TAURUS_E_INVALID, "null descriptor");
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
    if (!d->out) fail(TAURUS_E_INVALID, "out is null");
    if (d->out_on_host != 0) fail(TAURUS_E_INVALID, "out_on_host=%d is not supported by this build", d->out_on_host);
    if (d->hbm_budget < 0) fail(TAURUS_E_INVALID, "hbm_budget < 0");
}

static bool same_graph(const taurus_graph& a, const taurus_graph& b) {
    return a.n == b.n && a.e == b.e && a.row_off == b.row_off && a.col_dst == b.col_dst;
}

static void layer_init(taurus_layer* L) {
    const auto t_start = std::chrono::steady_clock::now();
    hipStream_t s = L->s;
    const taurus_graph& g = L->g;
    const taurus_layer_desc& d = L->d;
    const int64_t n = g.n, C = d.chunk;
    L->n = n;
    L->C = C;
    L->nchunks = ceil_div(n, C);
    L->d_o = d.d_out;
    L->ncols = d.agg == TAURUS_SAGE_MEAN ? 2 * d.d_out : d.d_out;
    row_group_shape(L->d_o, &L->G, &L->VEC);
    const int T = 256;

    // chunk index: shared from the plan for exact layers, else built here
    const taurus_plan* plan = d.plan;
    if (plan) {
        if (!same_graph(plan->g, g) || plan->chunk != C)
            fail(TAURUS_E_INVALID, "plan was built for another graph or chunk size");
        L->idx = plan->idx;
    } else {
        L->idx = build_index(g, C, L->mask, s, 0);
        L->ms_index = L->idx->ms_build;
    }
    const ChunkIndex& idx = *L->idx;

    L->cnt = L->arena.alloc<int2>(n, "pending counts");
    k_init_counts<<<(unsigned)ceil_div(n, T), T, 0, s>>>(idx.items_per_v, n, L->cnt);
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

    // working buffers
    L->acc = L->arena.alloc<float>(n * (int64_t)L->d_o, "accumulators");
    L->Y = L->arena.alloc<float>(std::min<int64_t>(C, n) * (int64_t)L->ncols, "chunk transform");
    const int64_t slots = std::max<int64_t>(1, idx.max_long_per_chunk);
    L->carry = L->arena.alloc<float>(slots * L->d_o, "hub piece carries");
    L->carry_cnt = L->arena.alloc<int32_t>(slots, "hub piece counts");
    L->pushed.assign((size_t)L->nchunks, 0);
    if (d.profile) {  // four events per chunk: before/after transform, scatter, fix-up
        L->events.assign((size_t)L->nchunks * 4, nullptr);
        for (auto& ev : L->events) TAURUS_HIP(hipEventCreate(&ev));
    }
    // host-side copies above read pageable memory that must stay valid until they ran
    TAURUS_HIP(hipStreamSynchronize(s));
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
    const ChunkIndex& idx = *L->idx;
    hipStream_t s = L->s;
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    if (L->d.profile) {
        for (int i = 0; i < 4; i++) ev[i] = L->events[(size_t)k * 4 + i];
        TAURUS_HIP(hipEventRecord(ev[0], s));
    }
    L->pushed[(size_t)k] = 1;
    L->npushed++;
    gemm_f32(static_cast<const float*>(x), e - b, L->d.d_in, L->wpack, L->ncols, L->n_out ? L->n_out + b : nullptr,
             L->Y, s);
    if (ev[1]) TAURUS_HIP(hipEventRecord(ev[1], s));
    ScatterParams p;
    p.Y = L->Y;
    p.ystride = L->ncols;
    p.self_col = L->d.agg == TAURUS_SAGE_MEAN ? L->d_o : 0;
    p.src = idx.item_src + idx.chunk_off[(size_t)k];
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
    p.long_base = idx.long_off[(size_t)k];
    const int64_t ns = idx.short_off[(size_t)k + 1] - idx.short_off[(size_t)k];
    const int64_t nl = idx.long_off[(size_t)k + 1] - idx.long_off[(size_t)k];
    if (ns + nl > 0)
        dispatch_scatter(L->G, L->VEC, p, idx.u_short + idx.short_off[(size_t)k], ns,
                         idx.u_long + idx.long_off[(size_t)k], nl, s);
    if (ev[2]) TAURUS_HIP(hipEventRecord(ev[2], s));
    const int64_t nfix = idx.fix_off[(size_t)k + 1] - idx.fix_off[(size_t)k];
    if (nfix > 0) dispatch_fixup(L->G, L->VEC, p, idx.u_fix + idx.fix_off[(size_t)k], nfix, s);
    if (ev[3]) TAURUS_HIP(hipEventRecord(ev[3], s));
}

static int finalize(taurus_layer* L, taurus_stats* st) {
    if (L->poisoned) fail(TAURUS_E_STATE, "layer handle is poisoned by an earlier failure");
    hipStream_t s = L->s;
    const ChunkIndex& idx = *L->idx;
    Arena tmp(s);
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
        st->messages = idx.kept;
        st->self_terms = L->n;
        st->pairs = idx.pairs;
        st->pending_left = (int64_t)left;
        st->completed = L->n - (int64_t)left;
        st->chunks = L->nchunks;
        st->chunks_pushed = L->npushed;
        st->short_units = idx.n_short;
        st->wave_units = idx.n_long;
        st->split_segments = idx.n_fix;
        st->device_bytes = L->arena.peak() + (L->ms_index > 0 ? idx.arena.peak() : 0);
        st->ms_init = L->ms_init;
        for (size_t i = 0; i + 3 < L->events.size(); i += 4) {
            const size_t k = i / 4;
            if (!L->pushed[k]) continue;
            float a = 0, b = 0, c = 0;
            TAURUS_HIP(hipEventElapsedTime(&a, L->events[i], L->events[i + 1]));
            TAURUS_HIP(hipEventElapsedTime(&b, L->events[i + 1], L->events[i + 2]));
            TAURUS_HIP(hipEventElapsedTime(&c, L->events[i + 2], L->events[i + 3]));
            st->ms_gemm += a;
            st->ms_scatter += b;
            st->ms_fixup += c;
            st->launches_gemm++;
            st->launches_scatter += (idx.short_off[k + 1] > idx.short_off[k] || idx.long_off[k + 1] > idx.long_off[k]) ? 1 : 0;
            st->launches_fixup += idx.fix_off[k + 1] > idx.fix_off[k] ? 1 : 0;
        }
    }
    return left ? TAURUS_E_INCOMPLETE : TAURUS_OK;
}

}  // namespace taurus

// ------------------------------------------------------------------ C ABI --

using namespace taurus;

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
    try {
        return build_csr_impl(n, e, src, dst, row_off, col_dst, static_cast<hipStream_t>(stream));
    } catch (const Failure& f) {
        return f.status;
    } catch (const std::exception& x) {
        set_error("internal error: %s", x.what());
        return TAURUS_E_DEVICE;
    }
}

int taurus_plan_create(const taurus_graph* g, int64_t chunk, void* stream, taurus_plan** out) {
    if (!out) {
        set_error("out handle pointer is null");
        return TAURUS_E_INVALID;
    }
    *out = nullptr;
    try {
        check_graph_args(g);
        if (chunk <= 0 || chunk >= ((int64_t)1 << 31)) fail(TAURUS_E_INVALID, "chunk %lld", (long long)chunk);
        auto P = std::make_unique<taurus_plan>();
        P->g = *g;
        P->chunk = chunk;
        P->idx = build_index(*g, chunk, nullptr, static_cast<hipStream_t>(stream), 0);
        *out = P.release();
        return TAURUS_OK;
    } catch (const Failure& f) {
        return f.status;
    } catch (const std::exception& x) {
        set_error("internal error: %s", x.what());
        return TAURUS_E_DEVICE;
    }
}

void taurus_plan_destroy(taurus_plan* P) { delete P; }

int taurus_layer_init(const taurus_graph* g, const taurus_layer_desc* d, taurus_layer** out) {
    if (!out) {
        set_error("out handle pointer is null");
        return TAURUS_E_INVALID;
    }
    *out = nullptr;
    taurus_layer* L = nullptr;
    try {
        check_graph_args(g);
        validate_desc(d);
        L = new taurus_layer();
        L->g = *g;
        L->d = *d;
        L->s = static_cast<hipStream_t>(d->stream);
        L->arena.set_stream(L->s);
        L->arena.set_budget(d->hbm_budget);
        layer_init(L);
        *out = L;
        return TAURUS_OK;
    } catch (const Failure& f) {
        if (L) (void)hipStreamSynchronize(L->s);
        delete L;
        return f.status;
    } catch (const std::exception& x) {
        if (L) (void)hipStreamSynchronize(L->s);
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
        taurus_stats local;
        taurus_stats* st = stats ? stats : &local;
        int rc = finalize(L, st);
        if (rc == TAURUS_E_INCOMPLETE)
            set_error("%lld destinations still have pending messages", (long long)st->pending_left);
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
    try {
        const int64_t words = ceil_div(L->g.e, 64);
        if (L->mask) {
            TAURUS_HIP(hipMemcpyAsync(mask_bits_host, L->mask, (size_t)words * 8, hipMemcpyDeviceToHost, L->s));
            TAURUS_HIP(hipStreamSynchronize(L->s));
        } else {
            for (int64_t w = 0; w < words; w++) mask_bits_host[w] = ~0ull;
            if (L->g.e % 64) mask_bits_host[words - 1] = (1ull << (L->g.e % 64)) - 1;
        }
        if (n_kept) *n_kept = L->idx->kept;
        return TAURUS_OK;
    } catch (const Failure& f) {
        return f.status;
    }
}

void taurus_layer_destroy(taurus_layer* L) {
    if (!L) return;
    (void)hipStreamSynchronize(L->s);
    delete L;
}

}  // extern "C"
