// One GNN layer as source-centric broadcast (Taurus, Sec. 3.1-3.6).
//
// Per graph and chunk size (the chunk index, shared by exact layers):
//   - the propagated in-edges (u, v), stably sorted by (chunk of the source,
//     v): in chunk j the messages to one destination form one contiguous
//     segment, sources ascending;
//   - each vertex's arrival count |M(v)| + 1: every propagated in-edge and
//     the self message count once (Sec. 3.4: O(|V|) pending counts; a vertex
//     completes when its count reaches zero);
//   - degree-bucketed work units: segments of 1, 2, 3-4 and 5-8 messages form
//     four short classes, each reduced by a row-group of lanes with a loop of
//     fixed length; longer segments are cut into pieces of at most PIECE_LEN
//     messages, each reduced by a whole wave; a segment cut into several
//     pieces (a hub) is completed by the fix-up pass, which sums the pieces'
//     partial rows in a fixed order.
// Per chunk (taurus_push_chunk):
//   1. transform: Y = X_c W on the matrix cores (GCN rows scaled by
//      d^_out(u)^-1/2; GraphSAGE Y = [X_c W_agg^T | X_c W_self^T]);
//   2. self pass: every vertex of the chunk adds its self row (the vertex's
//      own message: the W_self half for GraphSAGE, its normalised row for
//      GCN) to its accumulator -- a streaming pass over consecutive rows;
//      a vertex with a segment from its own chunk takes it in that
//      segment's flush instead, and in-core GraphSAGE layers add the others'
//      in the transform (step 1), leaving the pass only their counts;
//   3. scatter: per unit, the sum of its source rows scaled once by
//      1/|M(v)| (the per-message normalisation of Sec. 3.4 applied to the
//      segment sum) is added to v's fp32 accumulator; the pending count
//      drops by the segment length;
//   4. finalise in place: the flush that brings pending[v] to zero writes
//      out[v] = act(phi_v * acc[v] + b) directly (GCN phi_v = d^_in(v)^-1/2,
//      GraphSAGE phi_v = 1), the graduation step of Sec. 3.6;
//   5. fix-up: hub segments sum their pieces and flush the same way.
// A flush is the only writer of its destination within a kernel (segments
// of one chunk are disjoint, kernels of one layer are stream ordered), so
// accumulators are updated with plain loads and stores, no atomics.
#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <memory>
#include <mutex>
#include <thread>

#include "device.hpp"
#include "gemm_device.hpp"
#include "internal.hpp"
#include "resident.hpp"

namespace taurus {

int build_csr_impl(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                   int32_t* col_dst, hipStream_t s);
int build_csr_noalloc_impl(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                           int32_t* col_dst, hipStream_t s);
void gemm_f32(const float* X, int64_t M, int K, const float* Wp, int Nc, const float* rscale, float* Y,
              const SelfFlush* sf, hipStream_t s);
void gemm_pack_weights_f32(const float* W, int K, int Nc, std::vector<float>& packed);
void gemm_16(const uint16_t* X, int dtype, int64_t M, int K, const uint16_t* Wp, int Nc, const float* rscale,
             float* Y, const SelfFlush* sf, hipStream_t s);
void gemm_pack_weights_16(const float* W, int K, int Nc, int dtype, std::vector<uint16_t>& packed);
int gemm_packed_blocks_n(int nc);
const char* last_error_cstr();

constexpr int SC_THREADS = 256;
constexpr int NCLASS = 5;                           // short segment classes
constexpr int PIECE_LEN = 512;                      // longer segments: pieces of this many slots
constexpr int NOT_FIRST = 1 << 30;                  // unit.y flags (see seg_unit)
constexpr int SELF_HERE = 1 << 29;
constexpr int LEN_MASK = SELF_HERE - 1;
constexpr int NLIST = NCLASS + 2;                   // short classes, wave units, fix-up entries
constexpr int TALLY_SLOTS = 64;                     // spread of the self-message tallies
static_assert(RES_LISTS == NCLASS + 1, "residency walks the short classes and the wave units");

// most slots of a segment in short class c: 1, 2, 4, 8, 16
__host__ __device__ constexpr int class_len(int c) { return 1 << c; }

// ------------------------------------------------------------ init kernels --

// pending and expected arrival counts: |M(v)| propagated messages + 1 self
__global__ void k_init_counts(const int32_t* __restrict__ m, int64_t n, int2* __restrict__ cnt) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n) cnt[v] = make_int2(m[v] + 1, m[v] + 1);
}

// GCN source factor d^_out(u)^-1/2 with d^_out = out-degree + 1
__global__ void k_out_norm(const int64_t* __restrict__ row_off, int64_t n, float* __restrict__ n_out) {
    const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (u < n) n_out[u] = 1.0f / sqrtf((float)(row_off[u + 1] - row_off[u] + 1));
}

// the same for a sampled layer: the out-degree counts u's kept edges (set
// bits of the layer's mask over its CSR row)
// Kept out-edges of row u from the kept edges before each CSR position:
// before(i) = word_off[i / 64] + kept bits of mask word i / 64 below i.
__global__ void k_out_norm_kept(const int64_t* __restrict__ row_off, const uint64_t* __restrict__ mask,
                                const uint64_t* __restrict__ word_off, int64_t n, float* __restrict__ n_out) {
    const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (u >= n) return;
    auto before = [&](int64_t i) {
        const int64_t w = i >> 6;
        const int r = (int)(i & 63);
        return (int64_t)word_off[w] + (r ? __popcll(mask[w] & ((1ull << r) - 1ull)) : 0);
    };
    const int64_t kept = before(row_off[u + 1]) - before(row_off[u]);
    n_out[u] = 1.0f / sqrtf((float)(kept + 1));
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

// Chunk-index items of an exact layer.  CSR edge i (source u = the row
// containing i) becomes key (chunk(u) << vbits | v), value u - chunk(u)*C.
// A workgroup takes MI_TILE consecutive edges and finds their rows through
// tile_rows.
constexpr int MI_ITEMS = 16, MI_TILE = 256 * MI_ITEMS, MI_ROWS = 8192;
__global__ __launch_bounds__(256) void k_make_items(const int64_t* __restrict__ row_off,
                                                    const int32_t* __restrict__ col_dst, int64_t e, int64_t n,
                                                    int64_t C, int vbits, uint64_t* __restrict__ keys,
                                                    uint32_t* __restrict__ vals, int* __restrict__ bad) {
    __shared__ int32_t ro[MI_ROWS + 1];
    __shared__ int64_t bnd[2];
    const int64_t i0 = (int64_t)blockIdx.x * MI_TILE, i1 = min(i0 + MI_TILE, e);
    const TileRows t = tile_rows<MI_ROWS, MI_TILE>(row_off, n, i0, i1, ro, bnd);
    bool flag = false;
#pragma unroll 4
    for (int r = 0; r < MI_ITEMS; r++) {
        const int64_t i = i0 + (int64_t)r * 256 + threadIdx.x;
        if (i >= i1) break;
        bool later;
        const int64_t u = tile_row_of(t, row_off, ro, i0, i, later);
        const int64_t v = col_dst[i];
        // rows strictly ascending, no self loops (a simple graph)
        if (v == u || (later && col_dst[i - 1] >= v)) flag = true;
        const uint32_t cu = (uint32_t)u / (uint32_t)C;  // u < 2^31 and C < 2^31: 32-bit division
        keys[i] = ((uint64_t)cu << vbits) | (uint64_t)v;
        vals[i] = (uint32_t)u - cu * (uint32_t)C;
    }
    if (flag) atomicOr(bad, 4);
}

// propagated edges per mask word (bits at or past e are not edges)
__global__ void k_mask_word_counts(const uint64_t* __restrict__ mask, int64_t words, int64_t e,
                                   uint32_t* __restrict__ cnt) {
    const int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (w >= words) return;
    uint64_t m = mask[w];
    const int64_t left = e - w * 64;
    if (left < 64) m &= (1ull << left) - 1ull;
    cnt[w] = (uint32_t)__popcll(m);
}

// offs[j] = first sorted position whose chunk field (bits kshift and up) is
// >= j, j in [0, nchunks]
__global__ void k_chunk_bounds(const uint64_t* __restrict__ keys, int64_t total, int64_t nchunks, int kshift,
                               int64_t* __restrict__ offs) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j > nchunks) return;
    const uint64_t target = (uint64_t)j << kshift;
    int64_t lo = 0, hi = total;
    while (lo < hi) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (keys[mid] < target) lo = mid + 1;
        else hi = mid;
    }
    offs[j] = lo;
}

// Segment heads: item i < kept starts a new (chunk, destination) segment
// when i = 0 or its key differs from item i-1's.  Items are taken in tiles
// of HEAD_TILE: k_head_counts counts each tile's heads, and after a scan of
// the counts k_head_positions writes seg_start[s] = first item of segment
// s, in item order, and seg_start[P] = items.
constexpr int HEAD_ITEMS = 16;
constexpr int HEAD_TILE = 256 * HEAD_ITEMS;

__device__ inline bool seg_head(const uint64_t* keys, int64_t i, int64_t kept) {
    return i < kept && (i == 0 || keys[i] != keys[i - 1]);
}

__global__ __launch_bounds__(256) void k_head_counts(const uint64_t* __restrict__ keys,
                                                     const int64_t* __restrict__ kept,
                                                     uint64_t* __restrict__ counts) {
    __shared__ uint32_t wsum[4];
    const int64_t base = (int64_t)blockIdx.x * HEAD_TILE;
    const int64_t kp = *kept;
    uint32_t c = 0;
#pragma unroll
    for (int j = 0; j < HEAD_ITEMS; j++) c += seg_head(keys, base + (int64_t)j * 256 + threadIdx.x, kp) ? 1u : 0u;
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) c += __shfl_xor(c, d, 64);
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) counts[blockIdx.x] = (uint64_t)wsum[0] + wsum[1] + wsum[2] + wsum[3];
}

__global__ __launch_bounds__(256) void k_head_positions(const uint64_t* __restrict__ keys, int64_t items,
                                                        const int64_t* __restrict__ kept,
                                                        const uint64_t* __restrict__ tile_off, int64_t P,
                                                        int64_t* __restrict__ seg_start) {
    __shared__ uint8_t fl[HEAD_TILE];
    __shared__ uint32_t wsum[4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t base = (int64_t)blockIdx.x * HEAD_TILE;
    const int64_t kp = *kept;
#pragma unroll
    for (int j = 0; j < HEAD_ITEMS; j++) fl[j * 256 + tid] = seg_head(keys, base + (int64_t)j * 256 + tid, kp) ? 1 : 0;
    __syncthreads();
    // thread t ranks items [t*HEAD_ITEMS, (t+1)*HEAD_ITEMS) of the tile
    uint32_t c = 0;
#pragma unroll
    for (int j = 0; j < HEAD_ITEMS; j++) c += fl[tid * HEAD_ITEMS + j];
    uint32_t incl = c;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t y = __shfl_up(incl, d, 64);
        if (lane >= d) incl += y;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    uint64_t pos = tile_off[blockIdx.x] + incl - c;
    for (int w = 0; w < wave; w++) pos += wsum[w];
#pragma unroll
    for (int j = 0; j < HEAD_ITEMS; j++)
        if (fl[tid * HEAD_ITEMS + j] && pos < (uint64_t)P) seg_start[pos++] = base + tid * HEAD_ITEMS + j;
    if (blockIdx.x == 0 && tid == 0) seg_start[P] = items;
}

// work list of a segment: short class 0..NCLASS-1 by slot count, or NCLASS (wave pieces)
__device__ inline int seg_class(int64_t slots) {
#pragma unroll
    for (int c = 0; c < NCLASS; c++)
        if (slots <= class_len(c)) return c;
    return NCLASS;
}

// A segment's slots: its messages, plus the destination's self message when
// the segment comes from the destination's own chunk (it rides on that
// segment's flush as the last slot, one arrival).
__device__ inline int64_t seg_slots(int64_t len, uint32_t v, uint32_t chunk, int64_t C) {
    return len + (v / (uint32_t)C == chunk ? 1 : 0);
}

// Per segment: add its length to the destination's message count, note the
// destination's first chunk, mark a segment from the destination's own chunk
// (OWN_SEGMENT; it carries the self message) and record the segment's slot
// count.
// (COUNTED: the message counts and first chunks are known already, as for
// a sampled layer)
template <bool COUNTED>
__global__ void k_seg_classify(const uint64_t* __restrict__ keys, const int64_t* __restrict__ seg_start, int64_t P,
                               int vbits, int kshift, int64_t C, int32_t* __restrict__ m,
                               int32_t* __restrict__ first_chunk,
                               int32_t* __restrict__ slots_of, uint8_t* __restrict__ has_own,
                               unsigned long long* __restrict__ own_count) {
    const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (s >= P) return;
    const int64_t b = seg_start[s], len = seg_start[s + 1] - b;
    const uint64_t v = keys[b] & (((uint64_t)1 << vbits) - 1);
    const uint32_t chunk = (uint32_t)(keys[b] >> kshift);
    if (!COUNTED) {
        atomicAdd(&m[v], (int)len);
        atomicMin(&first_chunk[v], (int)chunk);
    }
    const int64_t slots = seg_slots(len, (uint32_t)v, chunk, C);
    if (slots > len) {
        has_own[v] = OWN_SEGMENT;
        atomicAdd(own_count, 1ull);
    }
    slots_of[s] = (int32_t)slots;
}

// What a unit of segment s says besides its slots: {first item relative to
// its chunk, NOT_FIRST, destination, SELF_HERE when the segment carries the
// self message}.  NOT_FIRST marks a segment that is not its destination's
// first flush when chunks are pushed in ascending order (the first flush is
// in the earlier of the first message chunk and the own chunk): its
// accumulator row then already holds a partial sum, so the scatter fetches
// the row together with the rows of its messages (the pending count still
// decides whether the row is used).
struct SegUnit {
    int64_t rel;
    int nf, v, self;
};
// Keys are (chunk << kshift | v); with kshift = vbits + 1 (sampled layers)
// bit vbits says the segment is not v's first flush, otherwise it comes
// from first_chunk.
__device__ inline SegUnit seg_unit(const uint64_t* keys, const int64_t* seg_start, int64_t s, int vbits, int kshift,
                                   int64_t C, const int64_t* chunk_off, const int32_t* first_chunk) {
    const int64_t b = seg_start[s];
    const uint64_t key = keys[b];
    SegUnit u;
    u.v = (int)(key & (((uint64_t)1 << vbits) - 1));
    const int chunk = (int)(key >> kshift);
    u.rel = b - chunk_off[chunk];
    const int own_chunk = (int)((uint32_t)u.v / (uint32_t)C);
    if (kshift > vbits)
        u.nf = (key >> vbits) & 1 ? NOT_FIRST : 0;
    else
        u.nf = chunk != min(first_chunk[u.v], own_chunk) ? NOT_FIRST : 0;
    u.self = own_chunk == chunk ? SELF_HERE : 0;
    return u;
}

// ---- work lists by tiles of segments ----
constexpr int LT_THREADS = 256, LT_PER = 16, LT_TILE = LT_THREADS * LT_PER;

// entries segment s adds to every list
__device__ inline void seg_entries(int64_t slots, int64_t (&c)[NLIST]) {
    const int cls = seg_class(slots);
    if (cls < NCLASS) {
        c[cls] += 1;
    } else {
        const int64_t pieces = (slots + PIECE_LEN - 1) / PIECE_LEN;
        c[NCLASS] += pieces;
        c[NCLASS + 1] += pieces > 1 ? 1 : 0;
    }
}

// tile_cnt[l * ntiles + t] = entries the segments of tile t add to list l
// (the tile's segments in LT_PER rounds of LT_THREADS consecutive ones)
__global__ __launch_bounds__(LT_THREADS) void k_list_tile_counts(const int32_t* __restrict__ slots_of, int64_t P,
                                                                int64_t ntiles, uint64_t* __restrict__ tile_cnt) {
    __shared__ int64_t part[LT_THREADS / 64][NLIST];
    int64_t c[NLIST] = {};
    const int64_t s0 = (int64_t)blockIdx.x * LT_TILE + threadIdx.x;
    for (int j = 0; j < LT_PER; j++)
        if (s0 + j * LT_THREADS < P) seg_entries(slots_of[s0 + j * LT_THREADS], c);
#pragma unroll
    for (int l = 0; l < NLIST; l++)
        for (int m = 32; m >= 1; m >>= 1) c[l] += __shfl_xor(c[l], m, 64);
    if ((threadIdx.x & 63) == 0)
        for (int l = 0; l < NLIST; l++) part[threadIdx.x >> 6][l] = c[l];
    __syncthreads();
    if (threadIdx.x < NLIST) {
        int64_t t = 0;
        for (int w = 0; w < LT_THREADS / 64; w++) t += part[w][threadIdx.x];
        tile_cnt[(int64_t)threadIdx.x * ntiles + blockIdx.x] = (uint64_t)t;
    }
}

// Units of tile t's segments, in segment order within each list, from the
// tile's positions tile_off[l * ntiles + t] (absolute in the work-list
// buffer).  The tile is taken in LT_PER rounds of LT_THREADS consecutive
// segments, one per thread, so reads and each list's writes are
// contiguous over the threads; a round's positions are a workgroup prefix
// of the entries its segments add (ballots for the one-entry lists, a scan
// for the wave pieces).  A segment that starts a chunk also writes, for
// that chunk and any empty chunks before it, each list's position there:
// dbases[l * (nchunks + 1) + k]; the last segment writes the list ends for
// the chunks after it and for k = nchunks.
__global__ __launch_bounds__(LT_THREADS) void k_list_emit(const uint64_t* __restrict__ keys,
                                                         const int64_t* __restrict__ seg_start,
                                                         const int32_t* __restrict__ slots_of, int64_t P,
                                                         int64_t ntiles, const uint64_t* __restrict__ tile_off,
                                                         int vbits, int kshift, int64_t C,
                                                         const int64_t* __restrict__ chunk_off,
                                                         const int32_t* __restrict__ first_chunk, int64_t nchunks,
                                                         int4* __restrict__ units, int64_t* __restrict__ dbases) {
    constexpr int NW = LT_THREADS / 64;
    __shared__ int64_t wsum[2][NW][NLIST];   // per round parity: entries of each wave
    __shared__ int64_t run[NLIST];           // list positions before the current round
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t lt = (1ull << lane) - 1ull;
    if (threadIdx.x < NLIST) run[threadIdx.x] = (int64_t)tile_off[(int64_t)threadIdx.x * ntiles + blockIdx.x];
    const int64_t t0 = (int64_t)blockIdx.x * LT_TILE;
    for (int r = 0; r < LT_PER; r++) {
        const int64_t sg = t0 + (int64_t)r * LT_THREADS + threadIdx.x;
        if (t0 + (int64_t)r * LT_THREADS >= P) break;  // uniform over the workgroup
        const int par = r & 1;
        const bool here = sg < P;
        const int64_t slots = here ? slots_of[sg] : 0;
        const int cls = here ? seg_class(slots) : -1;
        const int64_t pieces = cls == NCLASS ? (slots + PIECE_LEN - 1) / PIECE_LEN : 0;
        // this thread's entries before it in the wave, per list
        int64_t pre[NLIST];
#pragma unroll
        for (int l = 0; l < NCLASS; l++) {
            const uint64_t bal = __ballot(cls == l);
            pre[l] = __popcll(bal & lt);
            if (lane == 0) wsum[par][w][l] = __popcll(bal);
        }
        {
            const uint64_t bal = __ballot(pieces > 1);
            pre[NCLASS + 1] = __popcll(bal & lt);
            if (lane == 0) wsum[par][w][NCLASS + 1] = __popcll(bal);
        }
        int64_t x = pieces;
        if (__ballot(pieces > 0)) {  // uniform over the wave
            for (int m = 1; m < 64; m <<= 1) {
                const int64_t y = __shfl_up(x, m, 64);
                if (lane >= m) x += y;
            }
        }
        pre[NCLASS] = x - pieces;
        if (lane == 63) wsum[par][w][NCLASS] = x;
        __syncthreads();
#pragma unroll
        for (int l = 0; l < NLIST; l++) {
            int64_t before = run[l];
            for (int q = 0; q < w; q++) before += wsum[par][q][l];
            pre[l] += before;
        }
        if (here) {
            const int64_t b = seg_start[sg];
            const int64_t chunk = (int64_t)(keys[b] >> kshift);
            const int64_t prev = sg == 0 ? -1 : (int64_t)(keys[seg_start[sg - 1]] >> kshift);
            for (int64_t k = prev + 1; k <= chunk; k++)
                for (int l = 0; l < NLIST; l++) dbases[(int64_t)l * (nchunks + 1) + k] = pre[l];
            const SegUnit u = seg_unit(keys, seg_start, sg, vbits, kshift, C, chunk_off, first_chunk);
            if (cls < NCLASS) {
                units[pre[cls]] = make_int4((int)u.rel, (int)slots | u.nf | u.self, u.v, 0);
            } else {
                const int64_t first = pre[NCLASS];
                for (int q = 0; q < (int)pieces; q++) {
                    const int64_t o = (int64_t)q * PIECE_LEN;
                    const int plen = (int)min((int64_t)PIECE_LEN, slots - o);
                    const int self = q == pieces - 1 ? u.self : 0;
                    units[first + q] =
                        make_int4((int)(u.rel + o), plen | u.nf | self, u.v, pieces > 1 ? (int)(first + q) : -1);
                }
                if (pieces > 1) units[pre[NCLASS + 1]] = make_int4(u.v, (int)first, (int)pieces, 0);
            }
            if (sg == P - 1) {  // list ends for the chunks after the last segment's
                int64_t end[NLIST];
                for (int l = 0; l < NLIST; l++) end[l] = pre[l];
                if (cls < NCLASS) end[cls] += 1;
                else {
                    end[NCLASS] += pieces;
                    end[NCLASS + 1] += pieces > 1 ? 1 : 0;
                }
                for (int64_t k = chunk + 1; k <= nchunks; k++)
                    for (int l = 0; l < NLIST; l++) dbases[(int64_t)l * (nchunks + 1) + k] = end[l];
            }
        }
        // every thread has read run: add the round's totals (wsum[par] is
        // next written two rounds on, after the next round's barriers)
        __syncthreads();
        if (threadIdx.x < NLIST) {
            int64_t t = 0;
            for (int q = 0; q < NW; q++) t += wsum[par][q][threadIdx.x];
            run[threadIdx.x] += t;
        }
    }
}

// SELF_FIRST: v's own chunk is no later than its first message chunk, so
// with chunks pushed in ascending order its self message is its first flush
__global__ void k_self_first(const int32_t* __restrict__ first_chunk, int64_t n, int64_t C,
                             uint8_t* __restrict__ has_own) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n) has_own[v] = (has_own[v] & OWN_SEGMENT) | ((int64_t)first_chunk[v] >= v / C ? SELF_FIRST : 0);
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
    int y_bytes;           // bytes of Y addressable by the gathers (< 2^31)
    const int32_t* src;    // chunk items: local source row
    const uint8_t* has_own;  // per vertex: OWN_SEGMENT | SELF_FIRST
    int2* cnt;             // {pending, expected}
    float* acc;            // fp32 accumulator rows, d_o floats each
    const int32_t* slot;   // accumulator row of each vertex (residency pool), or null: row v
    int d_o;
    int agg;               // 0 GraphSAGE-mean, 1 GCN, 2 GIN
    int relu;
    int out_dtype;         // 0 fp32, 1 bf16, 2 fp16
    const float* bias;     // [d_o]
    void* out;             // [n][d_o]
    float* carry;          // per hub piece of the chunk: [d_o] partial contribution
    int32_t* carry_cnt;    // per hub piece: arrival count
    int64_t long_base;     // global index of the chunk's first wave unit (carry slot 0)
    int64_t first_row;     // first vertex of the chunk
    int64_t rows;          // vertices in the chunk
    // GAT aggregation only (k_scatter<G, VEC, true>): the weight of message
    // u -> v is exp(LeakyReLU(s_u + t_v) - m_v) / S_v, with s_u in column
    // d_o of u's row of Y, t_v = att_t[v * ystride], m_v = att_m[v] and
    // S_v = att_s[v]
    const float* att_t;
    const float* att_m;
    const float* att_s;
    // GIN with a perceptron (agg TAURUS_GIN_MLP): a completing destination's
    // hidden row ReLU(acc + b1) replaces its accumulator row; the chunk's
    // graduation transform reads it from there
    // self_done: the chunk's transform took the self messages of the
    // vertices without a segment here (SelfFlush); the self pass only takes
    // their arrival off the count, and, with self_tally set, counts how many
    // of those self messages found nothing accumulated and how many were the
    // last arrival ([TALLY_SLOTS][2], summed at finalize)
    int self_done;
    unsigned long long* self_tally;
};

struct ChunkUnits {        // this chunk's slice of the short classes and wave units
    const int4* u[NCLASS + 1];
    int64_t n[NCLASS + 1];
    // Row-group work of the short classes (longest first) and the self pass
    // is one sequence of batches laid after the row-groups the wave pieces
    // occupy; phase c starts at rot[c] of it (rot[NCLASS]: the self pass), so
    // on a small chunk the phases run side by side on different row-groups
    // instead of one after another on every row-group.
    int64_t rot[NCLASS + 1];
};

// First batch of a phase starting at `rot` of the row-group sequence for
// row-group gid of `stride` (the batches of gid are those congruent to gid).
__device__ inline int64_t phase_first(int64_t gid, int64_t rot, int64_t stride) {
    const int64_t d = (gid - rot) % stride;
    return d < 0 ? d + stride : d;
}

__device__ inline float4 f4_zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
__device__ inline float4 f4_add(float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); }
__device__ inline float4 f4_axpy(float s, float4 a, float4 b) {
    return make_float4(fmaf(s, a.x, b.x), fmaf(s, a.y, b.y), fmaf(s, a.z, b.z), fmaf(s, a.w, b.w));
}
__device__ inline float4 f4_scale(float s, float4 a) { return make_float4(s * a.x, s * a.y, s * a.z, s * a.w); }

__device__ inline float* acc_row(const ScatterParams& p, int v) {
    return p.acc + (int64_t)(p.slot ? p.slot[v] : v) * p.d_o;
}

// GAT: LeakyReLU slope of the attention scores, and the attention weight of
// the message from local row r of the chunk to v
constexpr float ATT_SLOPE = 0.2f;
__device__ inline float att_weight(const ScatterParams& p, int r, int v) {
    const float e0 = p.Y[(int64_t)r * p.ystride + p.d_o] + p.att_t[(int64_t)v * p.ystride];
    const float e = e0 > 0.f ? e0 : ATT_SLOPE * e0;
    return expf(e - p.att_m[v]) / p.att_s[v];
}

// weight of a message slot: GraphSAGE-mean 1/|M(v)| (|M(v)| = expected - 1),
// GCN 1 (sources are pre-scaled); the self slot always weighs 1
__device__ inline float seg_scale(int agg, int expect) {
    return agg == 0 ? (expect > 1 ? 1.0f / (float)(expect - 1) : 0.0f) : 1.0f;
}

// Rows in flight per row-group: 16 slots of up to two float4 per lane, 8 of
// four; half as many in the lean build (twice the waves per SIMD, for
// chunks with too little work to hide the latency of a batch).
__host__ __device__ constexpr int slots_per_round(int vec, bool lean = false) {
    return (vec <= 2 ? 16 : 8) >> (lean ? 1 : 0);
}

// Units of short class `len` a row-group takes at once: their rows plus
// one early accumulator row each stay within 20 rows of up to two float4
// per lane (10 of four), and at most 8 units.
__host__ __device__ constexpr int batch_units(int vec, int len, bool lean = false) {
    const int k = ((vec <= 2 ? 20 : 10) >> (lean ? 1 : 0)) / (len + 1);
    return k < 1 ? 1 : (k > 8 ? 8 : k);
}

// vertices per row-group batch of the self pass
__host__ __device__ constexpr int self_batch_rows(int vec, bool lean = false) {
    return (vec <= 2 ? 8 : 4) >> (lean ? 1 : 0);
}

// Gathers of rows of the chunk transform go through a buffer resource: a
// slot is the 32-bit byte offset of its row in Y, and an offset past the end
// of Y (NO_ROW, an empty slot) reads as zeros, so no load is predicated.  A
// lane reads columns (j*G + lane)*4 .. +3 of the row for j < VEC; a lane
// whose columns are at or past d_o (widths that do not fill G*VEC float4)
// takes NO_ROW's offset instead and reads zeros.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
constexpr uint32_t NO_ROW = 0x7fffff00u;   // > any y_bytes; NO_ROW + a row's bytes stays below 2^32

__device__ inline __amdgpu_buffer_rsrc_t y_rsrc(const ScatterParams& p) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)p.Y, (short)0, p.y_bytes, 0x00020000);
}

// byte offset of local row r's message half, and of its self half
__device__ inline uint32_t msg_off(const ScatterParams& p, int r) { return (uint32_t)r * (uint32_t)(p.ystride * 4); }
__device__ inline uint32_t self_off(const ScatterParams& p, int r) {
    return (uint32_t)r * (uint32_t)(p.ystride * 4) + (uint32_t)p.self_col * 4u;
}

// Row at byte offset off (NO_ROW: zeros); qv = float4 per row that hold
// values: the lanes past them (a width that does not fill the row-group's
// G * VEC float4) load nothing, so a narrow row costs only its own bytes.
template <int G, int VEC>
__device__ inline void gather_row(__amdgpu_buffer_rsrc_t rs, uint32_t off, int lane, int qv, float4 (&r)[VEC]) {
    const uint32_t o = off + (uint32_t)lane * 16u;
#pragma unroll
    for (int j = 0; j < VEC; j++) {
        const uint32_t oj = (j * G + lane < qv) ? o : NO_ROW;
        const u32x4_t q = __builtin_amdgcn_raw_buffer_load_b128(rs, oj, j * G * 16, 0);
        r[j] = make_float4(__uint_as_float(q.x), __uint_as_float(q.y), __uint_as_float(q.z), __uint_as_float(q.w));
    }
}

template <int G, int VEC>
__device__ inline void load_acc_row(const ScatterParams& p, int v, int lane, float4 (&r)[VEC]) {
    const float* arow = acc_row(p, v);
#pragma unroll
    for (int j = 0; j < VEC; j++) {
        const int col = (j * G + lane) * 4;
        r[j] = col < p.d_o ? *reinterpret_cast<const float4*>(arow + col) : f4_zero();
    }
}

// Sole-owner flush of contribution c (already weighted) carrying `count`
// arrivals to v.  pe = {pending, expected} as read before the flush.  pre
// holds v's accumulator row if it was fetched early (have_pre).
template <int G, int VEC>
__device__ inline void flush_owner(const ScatterParams& p, int v, int2 pe, const float4 (&c)[VEC], int count,
                                   int lane, const float4 (&pre)[VEC], bool have_pre) {
    const int left = pe.x - count;
    const bool fresh = pe.x == pe.y;  // nothing accumulated yet: acc[v] is logically zero
    float4 t[VEC];
#pragma unroll
    for (int j = 0; j < VEC; j++) t[j] = c[j];
    if (!fresh) {
        float4 a[VEC];
        if (have_pre) {
#pragma unroll
            for (int j = 0; j < VEC; j++) a[j] = pre[j];
        } else {
            load_acc_row<G, VEC>(p, v, lane, a);
        }
#pragma unroll
        for (int j = 0; j < VEC; j++) t[j] = f4_add(a[j], t[j]);
    }
    if (left == 0 && p.agg == TAURUS_GIN_MLP) {
        float* arow = acc_row(p, v);
#pragma unroll
        for (int j = 0; j < VEC; j++) {
            const int col = (j * G + lane) * 4;
            if (col < p.d_o) {
                const float4 b = *reinterpret_cast<const float4*>(p.bias + col);
                float4 z = f4_add(t[j], b);
                z.x = fmaxf(z.x, 0.f); z.y = fmaxf(z.y, 0.f);
                z.z = fmaxf(z.z, 0.f); z.w = fmaxf(z.w, 0.f);
                *reinterpret_cast<float4*>(arow + col) = z;
            }
        }
    } else if (left == 0) {
        const float phi = p.agg == 1 ? 1.0f / sqrtf((float)pe.y) : 1.0f;
#pragma unroll
        for (int j = 0; j < VEC; j++) {
            const int col = (j * G + lane) * 4;
            if (col < p.d_o) {
                const float4 b = *reinterpret_cast<const float4*>(p.bias + col);
                float4 z = f4_axpy(phi, t[j], b);
                if (p.relu) {
                    z.x = fmaxf(z.x, 0.f); z.y = fmaxf(z.y, 0.f);
                    z.z = fmaxf(z.z, 0.f); z.w = fmaxf(z.w, 0.f);
                }
                store_out4(p.out, p.out_dtype, (int64_t)v * p.d_o + col, z);
            }
        }
    } else {
        float* arow = acc_row(p, v);
#pragma unroll
        for (int j = 0; j < VEC; j++) {
            const int col = (j * G + lane) * 4;
            if (col < p.d_o) *reinterpret_cast<float4*>(arow + col) = t[j];
        }
    }
    if (lane == 0) p.cnt[v].x = left;
}

// Value of `reg[k / G]` held by lane k % G of this row-group (k < NREG * G).
template <int G, int NREG>
__device__ inline int rg_pick(const int (&reg)[NREG], int k) {
    int r = 0;
#pragma unroll
    for (int q = 0; q < NREG; q++) {
        const int t = __shfl(reg[q], k % G, G);
        if (k / G == q) r = t;
    }
    return r;
}

// Short class of segments of at most LEN slots (messages plus the self
// slot of an own-chunk segment).  A row-group takes K consecutive units of
// the class at a time, K*LEN slots in all, so that up to 16 rows plus the
// accumulator rows of the K destinations are in flight at once.  Loads are
// spread over the row-group's lanes (descriptor k in lane k % G, slot j's
// row offset in lane j % G) and shared by shuffles.  Slot 0 of a unit with
// SELF_HERE is the destination's own row (weight 1), its other slots are
// messages (weight sigma_v).  Software-pipelined: the next batch's row
// offsets and the descriptors after it are requested while this batch's
// rows are in flight.
template <int G, int VEC, int LEN, bool ATT, bool LEAN>
__device__ inline void short_batches(const ScatterParams& p, const int4* __restrict__ units, int64_t n, int64_t rot) {
    constexpr int SLOTS = slots_per_round(VEC, LEAN);
    constexpr int K = batch_units(VEC, LEN, LEAN);                            // units per batch
    constexpr int TS = K * LEN;                                               // slots per batch
    constexpr int RB = TS < SLOTS ? TS : SLOTS;                               // rows per round
    static_assert(TS <= SLOTS || K == 1, "a batch of several units fits one round");
    constexpr int KD = (K + G - 1) / G;                                       // descriptor registers
    constexpr int CR = (TS + G - 1) / G;                                      // offset registers
    constexpr int NRG = SC_THREADS / G;
    const int rg = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t nb = (n + K - 1) / K;
    const int64_t stride = (int64_t)gridDim.x * NRG;
    int64_t b = phase_first((int64_t)blockIdx.x * NRG + rg, rot, stride);
    if (b >= nb) return;  // the whole row-group
    const __amdgpu_buffer_rsrc_t rs = y_rsrc(p);
    const int qv = p.d_o >> 2;  // float4 of a row that hold values

    // descriptor k of batch bb in lane k % G, register k / G; an empty unit
    // has no slots and v = -1
    auto load_desc = [&](int64_t bb, int (&dx)[KD], int (&dy)[KD], int (&dv)[KD]) {
#pragma unroll
        for (int q = 0; q < KD; q++) {
            const int k = q * G + lane;
            const int64_t u = bb * K + k;
            int4 w = make_int4(0, 0, -1, 0);
            if (k < K && bb < nb && u < n) w = units[u];
            dx[q] = w.x;
            dy[q] = w.y;
            dv[q] = w.z;
        }
    };
    // slot j = (unit j / LEN, position j % LEN) of the batch in lane j % G
    // (with ATT, its attention weight beside it)
    auto load_offsets = [&](const int (&dx)[KD], const int (&dy)[KD], const int (&dv)[KD], uint32_t (&off)[CR],
                            float (&wt)[CR]) {
#pragma unroll
        for (int q = 0; q < CR; q++) {
            const int j = q * G + lane;
            const int k = j / LEN, i = j % LEN;
            const int x = rg_pick<G, KD>(dx, k), y = rg_pick<G, KD>(dy, k), v = rg_pick<G, KD>(dv, k);
            const int self = (y & SELF_HERE) ? 1 : 0;
            const int slots = y & LEN_MASK;
            uint32_t o = NO_ROW;
            if (j < TS && i < slots) {
                if (self && i == 0) o = self_off(p, (int)((int64_t)v - p.first_row));
                else o = msg_off(p, p.src[x + i - self]);
            }
            off[q] = o;
            if constexpr (ATT) {
                float a = 0.f;
                if (j < TS && i < slots)
                    a = att_weight(p, (self && i == 0) ? (int)((int64_t)v - p.first_row) : p.src[x + i - self], v);
                wt[q] = a;
            }
        }
    };

    int dx[KD], dy[KD], dv[KD];
    uint32_t off[CR];
    float wt[CR];
    load_desc(b, dx, dy, dv);
    load_offsets(dx, dy, dv, off, wt);
    int64_t b1 = b + stride;
    int nx[KD], ny[KD], nv[KD];
    load_desc(b1, nx, ny, nv);
    for (;;) {
        // this batch's rows (the first round of them), counts and early
        // accumulator rows
        float4 rows[RB][VEC];
        uint32_t so[TS];
#pragma unroll
        for (int j = 0; j < TS; j++) so[j] = (uint32_t)__shfl((int)off[j / G], j % G, G);
        float sw[TS];
        if constexpr (ATT) {
#pragma unroll
            for (int j = 0; j < TS; j++) sw[j] = __shfl(wt[j / G], j % G, G);
        }
#pragma unroll
        for (int j = 0; j < RB; j++) gather_row<G, VEC>(rs, so[j], lane, qv, rows[j]);
        int2 pe_l[KD];
#pragma unroll
        for (int q = 0; q < KD; q++) pe_l[q] = dv[q] >= 0 ? p.cnt[dv[q]] : make_int2(0, 0);
        int uy[K], uv[K];
        float4 pre[K][VEC];
#pragma unroll
        for (int k = 0; k < K; k++) {
            uy[k] = __shfl(dy[k / G], k % G, G);
            uv[k] = __shfl(dv[k / G], k % G, G);
            if (uv[k] >= 0 && (uy[k] & NOT_FIRST)) load_acc_row<G, VEC>(p, uv[k], lane, pre[k]);
        }
        // next batch's row offsets, and the descriptors of the one after
        const bool more = b1 < nb;
        uint32_t noff[CR];
        float nwt[CR];
#pragma unroll
        for (int q = 0; q < CR; q++) {
            noff[q] = NO_ROW;
            nwt[q] = 0.f;
        }
        if (more) load_offsets(nx, ny, nv, noff, nwt);
        const int64_t b2 = b1 + stride;
        int mx[KD], my[KD], mv[KD];
        load_desc(b2, mx, my, mv);
        // sum and flush each unit of this batch
#pragma unroll
        for (int k = 0; k < K; k++) {
            int2 pe;
            pe.x = __shfl(pe_l[k / G].x, k % G, G);
            pe.y = __shfl(pe_l[k / G].y, k % G, G);
            const float sig = seg_scale(p.agg, pe.y);
            float w0 = (uy[k] & SELF_HERE) ? 1.0f : sig;  // slot 0: own row or a message
            if constexpr (ATT) w0 = sw[k * LEN];
            float4 sa[VEC], c[VEC];
#pragma unroll
            for (int jv = 0; jv < VEC; jv++) {
                sa[jv] = f4_zero();
                c[jv] = f4_scale(w0, rows[(k * LEN) % RB][jv]);
            }
#pragma unroll
            for (int i = 1; i < LEN; i++) {
                const int j = k * LEN + i;
                if (j >= RB && j % RB == 0) {  // next round (a single-unit batch)
#pragma unroll
                    for (int jj = 0; jj < RB; jj++) gather_row<G, VEC>(rs, so[j + jj], lane, qv, rows[jj]);
                }
                if constexpr (ATT) {
#pragma unroll
                    for (int jv = 0; jv < VEC; jv++) c[jv] = f4_axpy(sw[j], rows[j % RB][jv], c[jv]);
                } else {
#pragma unroll
                    for (int jv = 0; jv < VEC; jv++) sa[jv] = f4_add(sa[jv], rows[j % RB][jv]);
                }
            }
            if (uv[k] < 0) continue;
            if constexpr (!ATT) {
#pragma unroll
                for (int jv = 0; jv < VEC; jv++) c[jv] = f4_axpy(sig, sa[jv], c[jv]);
            }
            flush_owner<G, VEC>(p, uv[k], pe, c, uy[k] & LEN_MASK, lane, pre[k], (uy[k] & NOT_FIRST) != 0);
        }
        if (!more) break;
        b = b1;
        b1 = b2;
#pragma unroll
        for (int q = 0; q < KD; q++) {
            dx[q] = nx[q]; dy[q] = ny[q]; dv[q] = nv[q];
            nx[q] = mx[q]; ny[q] = my[q]; nv[q] = mv[q];
        }
#pragma unroll
        for (int q = 0; q < CR; q++) {
            off[q] = noff[q];
            wt[q] = nwt[q];
        }
    }
}

// Wave units (pieces of at most PIECE_LEN slots of the longer segments): one
// per wave.  The piece's message row offsets are loaded at once, one per
// lane and register (message i in lane i % 64, register i / 64), and handed
// out by shuffles; each round every row-group gathers SLOTS rows.  A piece
// with SELF_HERE (the last piece of an own-chunk segment) holds the
// destination's own row as its last slot, fetched by row-group 0 beside the
// rounds.  The row-groups' partial sums are combined with cross-lane
// shuffles and row-group 0 flushes (or parks the partial row of a hub piece
// in its carry slot).  The next piece's descriptor is fetched ahead and its
// offsets are requested while the first round's rows are in flight.
template <int G, int VEC, bool ATT, bool LEAN>
__device__ inline void wave_pieces(const ScatterParams& p, const int4* __restrict__ units, int64_t n) {
    constexpr int SLOTS = slots_per_round(VEC, LEAN);
    constexpr int NREG = PIECE_LEN / 64;
    const int wave = threadIdx.x >> 6, l64 = threadIdx.x & 63;
    const int rg = l64 / G, lane = l64 % G;
    const int64_t wstride = (int64_t)gridDim.x * (SC_THREADS / 64);
    int64_t un = (int64_t)blockIdx.x * (SC_THREADS / 64) + wave;
    if (un >= n) return;  // the whole wave
    const __amdgpu_buffer_rsrc_t rs = y_rsrc(p);
    const int qv = p.d_o >> 2;  // float4 of a row that hold values
    auto load_offsets = [&](int4 w, uint32_t (&cr)[NREG], float (&wt)[NREG]) {
        const int items = (w.y & LEN_MASK) - ((w.y & SELF_HERE) ? 1 : 0);
#pragma unroll
        for (int t = 0; t < NREG; t++) {
            const int i = t * 64 + l64;
            cr[t] = i < items ? msg_off(p, p.src[w.x + i]) : NO_ROW;
            if constexpr (ATT) wt[t] = i < items ? att_weight(p, p.src[w.x + i], w.z) : 0.f;
        }
    };
    int4 w = units[un];
    uint32_t cr[NREG];
    float wt[NREG];
    load_offsets(w, cr, wt);
    int64_t un1 = un + wstride;
    int4 wn = un1 < n ? units[un1] : make_int4(0, 0, 0, 0);
    for (;;) {
        const int v = w.z, L = w.y & LEN_MASK;
        const bool self = (w.y & SELF_HERE) != 0;
        const int items = L - (self ? 1 : 0);
        const bool flush = w.w < 0;
        const int2 pe = p.cnt[v];
        float4 pre[VEC], srow[VEC];
        const bool have_pre = flush && rg == 0 && (w.y & NOT_FIRST);
        if (have_pre) load_acc_row<G, VEC>(p, v, lane, pre);
        gather_row<G, VEC>(rs, self && rg == 0 ? self_off(p, (int)((int64_t)v - p.first_row)) : NO_ROW, lane, qv, srow);
        const bool more = un1 < n;
        uint32_t ncr[NREG];
        float nwt[NREG];
#pragma unroll
        for (int t = 0; t < NREG; t++) {
            ncr[t] = NO_ROW;
            nwt[t] = 0.f;
        }
        float4 sa[VEC];
#pragma unroll
        for (int jv = 0; jv < VEC; jv++) sa[jv] = f4_zero();
        // one round: SLOTS row offsets of this row-group -> rows -> sum
        // (with ATT, each row times its weight ow[k])
        auto round = [&](const uint32_t (&o)[SLOTS], const float (&ow)[SLOTS]) {
            float4 rows[SLOTS][VEC];
#pragma unroll
            for (int k = 0; k < SLOTS; k++) gather_row<G, VEC>(rs, o[k], lane, qv, rows[k]);
#pragma unroll
            for (int k = 0; k < SLOTS; k++)
#pragma unroll
                for (int jv = 0; jv < VEC; jv++) {
                    if constexpr (ATT) sa[jv] = f4_axpy(ow[k], rows[k][jv], sa[jv]);
                    else sa[jv] = f4_add(sa[jv], rows[k][jv]);
                }
        };
        const int nreg = (items + 63) / 64;
        bool first = true;
        if constexpr (G <= SLOTS) {
            // a round takes M registers: slot k of row-group rg is lane
            // G*rg + k % G of register k / G
            constexpr int M = SLOTS / G;
            for (int r = 0; r < nreg; r += M) {
                uint32_t o[SLOTS];
                float ow[SLOTS];
#pragma unroll
                for (int k = 0; k < SLOTS; k++) {
                    o[k] = (uint32_t)__shfl((int)cr[k / G], G * rg + k % G, 64);
                    if constexpr (ATT) ow[k] = __shfl(wt[k / G], G * rg + k % G, 64);
                }
                if (first && more) load_offsets(wn, ncr, nwt);
                first = false;
                round(o, ow);
#pragma unroll
                for (int t = 0; t < NREG; t++) {
                    cr[t] = t + M < NREG ? cr[t + M] : NO_ROW;
                    if constexpr (ATT) wt[t] = t + M < NREG ? wt[t + M] : 0.f;
                }
            }
        } else {
            // a register takes G / SLOTS rounds: slot k of row-group rg in
            // round h is lane G*rg + SLOTS*h + k
            constexpr int H = G / SLOTS;
            for (int r = 0; r < nreg; r++) {
#pragma unroll 1
                for (int h = 0; h < H; h++) {
                    uint32_t o[SLOTS];
                    float ow[SLOTS];
#pragma unroll
                    for (int k = 0; k < SLOTS; k++) {
                        o[k] = (uint32_t)__shfl((int)cr[0], G * rg + SLOTS * h + k, 64);
                        if constexpr (ATT) ow[k] = __shfl(wt[0], G * rg + SLOTS * h + k, 64);
                    }
                    if (first && more) load_offsets(wn, ncr, nwt);
                    first = false;
                    round(o, ow);
                }
#pragma unroll
                for (int t = 0; t < NREG; t++) {
                    cr[t] = t + 1 < NREG ? cr[t + 1] : NO_ROW;
                    if constexpr (ATT) wt[t] = t + 1 < NREG ? wt[t + 1] : 0.f;
                }
            }
        }
        if (first && more) load_offsets(wn, ncr, nwt);
        const int64_t un2 = un1 + wstride;
        const int4 wn2 = un2 < n ? units[un2] : make_int4(0, 0, 0, 0);
        float4 c[VEC];
        if constexpr (ATT) {
            // the self row (zeros unless SELF_HERE) times its attention
            const float as = self ? att_weight(p, (int)((int64_t)v - p.first_row), v) : 0.f;
#pragma unroll
            for (int jv = 0; jv < VEC; jv++) c[jv] = f4_axpy(as, srow[jv], sa[jv]);
        } else {
            const float sig = seg_scale(p.agg, pe.y);
#pragma unroll
            for (int jv = 0; jv < VEC; jv++) c[jv] = f4_axpy(sig, sa[jv], srow[jv]);
        }
#pragma unroll
        for (int d = G; d < 64; d <<= 1)
#pragma unroll
            for (int jv = 0; jv < VEC; jv++) {
                c[jv].x += __shfl_xor(c[jv].x, d, 64);
                c[jv].y += __shfl_xor(c[jv].y, d, 64);
                c[jv].z += __shfl_xor(c[jv].z, d, 64);
                c[jv].w += __shfl_xor(c[jv].w, d, 64);
            }
        if (rg == 0) {
            if (flush) {
                flush_owner<G, VEC>(p, v, pe, c, L, lane, pre, have_pre);
            } else {
                const int64_t slot = (int64_t)w.w - p.long_base;
                float* crow = p.carry + slot * p.d_o;
#pragma unroll
                for (int jv = 0; jv < VEC; jv++) {
                    const int col = (jv * G + lane) * 4;
                    if (col < p.d_o) *reinterpret_cast<float4*>(crow + col) = c[jv];
                }
                if (lane == 0) p.carry_cnt[slot] = L;
            }
        }
        if (!more) break;
        w = wn;
        wn = wn2;
        un1 = un2;
#pragma unroll
        for (int t = 0; t < NREG; t++) {
            cr[t] = ncr[t];
            wt[t] = nwt[t];
        }
    }
}

// Self pass over the chunk's own vertices without a segment from this
// chunk (the others take their self message in their segment's flush): one
// arrival each.  A row-group takes K consecutive vertices at a time --
// consecutive rows of Y and of the accumulators.  These vertices have no
// other flush in the launch.  When the transform has already added their
// self rows (self_done), only the counts are updated.
template <int G, int VEC, bool ATT, bool LEAN>
__device__ inline void self_batches(const ScatterParams& p, int64_t rot) {
    constexpr int K = self_batch_rows(VEC, LEAN);
    constexpr int KD = (K + G - 1) / G;
    constexpr int NRG = SC_THREADS / G;
    const int rg = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t nrg = (int64_t)gridDim.x * NRG;
    const int64_t stride = nrg * K;
    if (!ATT && p.self_done) {
        int fresh = 0, last = 0;
        for (int64_t r0 = phase_first((int64_t)blockIdx.x * NRG + rg, rot, nrg) * K; r0 < p.rows; r0 += stride) {
#pragma unroll
            for (int q = 0; q < KD; q++) {
                const int k = q * G + lane;
                const int64_t v = p.first_row + r0 + k;
                if (k < K && r0 + k < p.rows && !(p.has_own[v] & OWN_SEGMENT)) {
                    const int2 pe = p.cnt[v];
                    fresh += pe.x == pe.y;
                    last += pe.x == 1;
                    p.cnt[v].x = pe.x - 1;
                }
            }
        }
        if (p.self_tally) {
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) {
                fresh += __shfl_xor(fresh, o);
                last += __shfl_xor(last, o);
            }
            if ((threadIdx.x & 63) == 0 && (fresh | last)) {
                unsigned long long* t = p.self_tally + 2 * (blockIdx.x % TALLY_SLOTS);
                atomicAdd(t, (unsigned long long)fresh);
                atomicAdd(t + 1, (unsigned long long)last);
            }
        }
        return;
    }
    const __amdgpu_buffer_rsrc_t rs = y_rsrc(p);
    const int qv = p.d_o >> 2;  // float4 of a row that hold values
    for (int64_t r0 = phase_first((int64_t)blockIdx.x * NRG + rg, rot, nrg) * K; r0 < p.rows; r0 += stride) {
        int fl[KD];
        int2 pe_l[KD];
#pragma unroll
        for (int q = 0; q < KD; q++) {
            const int k = q * G + lane;
            const int64_t r = r0 + k;
            fl[q] = OWN_SEGMENT;  // nothing to do
            pe_l[q] = make_int2(0, 0);
            if (k < K && r < p.rows) {
                fl[q] = p.has_own[p.first_row + r];
                if (!(fl[q] & OWN_SEGMENT)) pe_l[q] = p.cnt[p.first_row + r];
            }
        }
        float4 rows[K][VEC], pre[K][VEC];
        int f[K];
#pragma unroll
        for (int k = 0; k < K; k++) {
            f[k] = rg_pick<G, KD>(fl, k);
            const bool todo = !(f[k] & OWN_SEGMENT);
            gather_row<G, VEC>(rs, todo ? self_off(p, (int)(r0 + k)) : NO_ROW, lane, qv, rows[k]);
            if (todo && !(f[k] & SELF_FIRST)) load_acc_row<G, VEC>(p, (int)(p.first_row + r0 + k), lane, pre[k]);
        }
#pragma unroll
        for (int k = 0; k < K; k++) {
            if (f[k] & OWN_SEGMENT) continue;
            int2 pe;
            pe.x = __shfl(pe_l[k / G].x, k % G, G);
            pe.y = __shfl(pe_l[k / G].y, k % G, G);
            if constexpr (ATT) {
                const float as = att_weight(p, (int)(r0 + k), (int)(p.first_row + r0 + k));
#pragma unroll
                for (int jv = 0; jv < VEC; jv++) rows[k][jv] = f4_scale(as, rows[k][jv]);
            }
            flush_owner<G, VEC>(p, (int)(p.first_row + r0 + k), pe, rows[k], 1, lane, pre[k],
                                !(f[k] & SELF_FIRST));
        }
    }
}

// Degree-bucketed scatter of one chunk, persistent: the grid is sized to
// what the GPU holds at once and walks the wave pieces (longest work
// first), the short classes from long to short, then the self pass.
// ATT: GAT's aggregation pass, every slot weighted by its attention.  The
// plain aggregation takes the lean row budget (half the rows in flight per
// row-group) and runs three waves per SIMD (two for rows of four float4
// per lane): more row-groups resident hide the dependent loads of a batch
// better than more rows per row-group do.  GAT's pass keeps the full
// budget and two waves (its weights need the registers).
template <int G, int VEC, bool ATT = false>
__global__ __launch_bounds__(SC_THREADS) __attribute__((amdgpu_waves_per_eu(ATT || VEC > 2 ? 2 : 3)))
void k_scatter(ScatterParams p, ChunkUnits cu) {
    constexpr bool LEAN = !ATT;
    wave_pieces<G, VEC, ATT, LEAN>(p, cu.u[NCLASS], cu.n[NCLASS]);
    short_batches<G, VEC, 16, ATT, LEAN>(p, cu.u[4], cu.n[4], cu.rot[4]);
    short_batches<G, VEC, 8, ATT, LEAN>(p, cu.u[3], cu.n[3], cu.rot[3]);
    short_batches<G, VEC, 4, ATT, LEAN>(p, cu.u[2], cu.n[2], cu.rot[2]);
    short_batches<G, VEC, 2, ATT, LEAN>(p, cu.u[1], cu.n[1], cu.rot[1]);
    short_batches<G, VEC, 1, ATT, LEAN>(p, cu.u[0], cu.n[0], cu.rot[0]);
    self_batches<G, VEC, ATT, LEAN>(p, cu.rot[NCLASS]);
}

// A hub segment's pieces occupy consecutive carry slots; their partial rows
// (the last one holding the self row of an own-chunk segment) are summed in
// slot order and flushed.  Workgroup blk of the fix-up takes SC_THREADS / G
// hub segments, one per row-group.
template <int G, int VEC>
__device__ __attribute__((always_inline)) inline void fixup_rows(const ScatterParams& p, const int4* __restrict__ fix, int64_t nfix, int64_t blk) {
    constexpr int NRG = SC_THREADS / G;
    const int rg = threadIdx.x / G, lane = threadIdx.x % G;
    const int64_t idx = blk * NRG + rg;
    if (idx >= nfix) return;
    const int4 f = fix[idx];
    const int v = f.x;
    const int64_t first = (int64_t)f.y - p.long_base;
    float4 c[VEC], pre[VEC];
#pragma unroll
    for (int j = 0; j < VEC; j++) c[j] = pre[j] = f4_zero();
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
    flush_owner<G, VEC>(p, v, p.cnt[v], c, count, lane, pre, false);
}
template <int G, int VEC>
__global__ __launch_bounds__(SC_THREADS) void k_fixup(ScatterParams p, const int4* __restrict__ fix, int64_t nfix) {
    fixup_rows<G, VEC>(p, fix, nfix, blockIdx.x);
}

// ------------------------------------------------------------- dispatch ---

// Scatter configuration: G lanes per row-group with VEC float4 per lane,
// and the persistent grid size.
struct ScatterShape {
    int G, VEC;
    int64_t max_blocks, max_blocks_att;  // workgroups resident at once, plain and GAT builds
};

static int env_int(const char* name, int dflt) {
    const char* v = getenv(name);
    return v && *v ? atoi(v) : dflt;
}

template <int G, int VEC, bool ATT>
static int64_t resident_blocks() {
    int dev = 0, cus = 0, per_cu = 0;
    TAURUS_HIP(hipGetDevice(&dev));
    TAURUS_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    TAURUS_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_scatter<G, VEC, ATT>, SC_THREADS, 0));
    return (int64_t)std::max(1, cus) * std::max(1, per_cu);
}

// Row-group shape for an output width: two float4 per lane where the width
// allows (fewer lanes per destination, more destinations per wave), at least
// 4 and at most 64 lanes.
static ScatterShape scatter_shape(int d_o) {
    const int q = (d_o + 3) / 4;
    int g = 4;
    while (g < 64 && g * 2 < q) g <<= 1;
    int vec = (q + g - 1) / g;
    if (vec == 3) vec = 4;
    if (vec > 4) {
        g = 64;
        vec = (q + 63) / 64;
        if (vec == 3) vec = 4;
    }
    ScatterShape sh;
    sh.G = g;
    sh.VEC = vec;
    sh.max_blocks = sh.max_blocks_att = 0;
    return sh;
}

// the shapes scatter_shape() yields for widths 4..1024
#define TAURUS_ROW_SHAPES(X) X(4, 1) X(4, 2) X(8, 2) X(16, 2) X(32, 2) X(64, 2) X(64, 4)

static void dispatch_scatter(const ScatterShape& sh, const ScatterParams& p, ChunkUnits cu, hipStream_t s,
                             bool att = false) {
    const int nrg = SC_THREADS / sh.G;
    // the row-group sequence: wave pieces' row-groups, then the short
    // classes from the longest, then the self pass
    const bool lean = !att;  // the row budget k_scatter<G, VEC, att> is built with
    int64_t t = cu.n[NCLASS] * (64 / sh.G);
    for (int c = NCLASS - 1; c >= 0; c--) {
        cu.rot[c] = t;
        t += ceil_div(cu.n[c], batch_units(sh.VEC, class_len(c), lean));
    }
    cu.rot[NCLASS] = t;
    t += ceil_div(p.rows, self_batch_rows(sh.VEC, lean));
    const int64_t blocks = std::max<int64_t>(1, std::min(ceil_div(t, nrg), att ? sh.max_blocks_att : sh.max_blocks));
#define TAURUS_CASE(g, v)                                                         \
    if (sh.G == g && sh.VEC == v) {                                               \
        if (att) k_scatter<g, v, true><<<(unsigned)blocks, SC_THREADS, 0, s>>>(p, cu); \
        else k_scatter<g, v><<<(unsigned)blocks, SC_THREADS, 0, s>>>(p, cu);      \
        TAURUS_CHECK_LAUNCH();                                                    \
        return;                                                                   \
    }
    TAURUS_ROW_SHAPES(TAURUS_CASE)
#undef TAURUS_CASE
    fail(TAURUS_E_INVALID, "unsupported row shape G=%d VEC=%d", sh.G, sh.VEC);
}

static int64_t scatter_resident_blocks(const ScatterShape& sh, bool att) {
#define TAURUS_CASE(g, v) \
    if (sh.G == g && sh.VEC == v) return att ? resident_blocks<g, v, true>() : resident_blocks<g, v, false>();
    TAURUS_ROW_SHAPES(TAURUS_CASE)
#undef TAURUS_CASE
    fail(TAURUS_E_INVALID, "unsupported row shape G=%d VEC=%d", sh.G, sh.VEC);
}

static void dispatch_fixup(const ScatterShape& sh, const ScatterParams& p, const int4* fix, int64_t nfix,
                           hipStream_t s) {
#define TAURUS_CASE(g, v)                                                                         \
    if (sh.G == g && sh.VEC == v) {                                                               \
        k_fixup<g, v><<<(unsigned)ceil_div(nfix, SC_THREADS / g), SC_THREADS, 0, s>>>(p, fix, nfix); \
        TAURUS_CHECK_LAUNCH();                                                                    \
        return;                                                                                   \
    }
    TAURUS_ROW_SHAPES(TAURUS_CASE)
#undef TAURUS_CASE
    fail(TAURUS_E_INVALID, "unsupported row shape G=%d VEC=%d", sh.G, sh.VEC);
}

// ---------------------------------------------- graduation transform (GIN) --
// A GIN layer with a perceptron apply leaves each completed destination's
// hidden row t_v = ReLU(acc_v + b1) in its accumulator row.  After the
// chunk's flushes, the rows that completed in it take the perceptron's
// second layer on the matrix cores: out[v] = act(t_v W2 + b2), written in
// the output type (Sec. 3.6 transforms graduated vertices in batches).
// Which rows those are is fixed by the chunk index (the last chunk that
// carries a message to v), so the lists are built once per layer and the
// scatter keeps no list of its own: a shared counter bumped by every
// completing destination serialises the scatter's waves.

__device__ inline void store_out1(void* out, int dtype, int64_t idx, float z) {
    if (dtype == 0) static_cast<float*>(out)[idx] = z;
    else static_cast<uint16_t*>(out)[idx] = (uint16_t)(dtype == 1 ? f32_to_bf16_bits(z) : f32_to_f16_bits(z));
}

struct GradRows {
    const int32_t* ids;
    const float* b2;
    void* out;
    int d_out, dtype, relu;
    __device__ inline auto row(int64_t r) const {
        const int64_t base = (int64_t)ids[r] * d_out;
        return [=](int col, float x) {
            float z = x + (b2 ? b2[col] : 0.0f);
            if (relu) z = fmaxf(z, 0.0f);
            store_out1(out, dtype, base + col, z);
        };
    }
};

constexpr int GRAD_NB = 8;   // 16-column blocks per workgroup (128 columns)

// The graduation transform of one chunk: out[ids[r]] = act(hidden[ids[r]] W2
// + b2) for the M destinations that complete in it.
__global__ __launch_bounds__(256) void k_graduate(const float* __restrict__ hidden, int d_h,
                                                  const float4* __restrict__ w2p, int nbp, int d_out,
                                                  const int32_t* __restrict__ ids, int64_t M,
                                                  const float* __restrict__ b2, void* out, int dtype, int relu) {
    __shared__ PanelLds<TAURUS_F32, GRAD_NB> lds;
    const int64_t ngy = (nbp + GRAD_NB - 1) / GRAD_NB;
    const int64_t tiles = (M + PANEL_ROWS - 1) / PANEL_ROWS * ngy;
    const GradRows epi{ids, b2, out, d_out, dtype, relu};
    for (int64_t t = blockIdx.x; t < tiles; t += gridDim.x)  // uniform over the workgroup
        gemm_panel_core<TAURUS_F32, GRAD_NB>(hidden, M, d_h, w2p, nbp, d_out, (int)(t / ngy), (int)(t % ngy), lds,
                                             [=](int64_t r) { return (int64_t)ids[r]; }, epi);
}

// The chunk a destination completes in is the last chunk that carries one
// of its messages: its own chunk (the self message) or a later one holding
// one of its segments.  k_own_chunk starts lc[v] at v's own chunk (and ids
// at the identity); k_unit_chunks raises it to the chunk of every work-list
// entry naming v, whose entries of chunk k sit at [offs[k], offs[k + 1]).
__global__ __launch_bounds__(256) void k_own_chunk(uint32_t* __restrict__ lc, uint32_t* __restrict__ ids, int64_t n,
                                                   int64_t C) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n) {
        lc[v] = (uint32_t)(v / C);
        ids[v] = (uint32_t)v;
    }
}

__global__ __launch_bounds__(256) void k_unit_chunks(const int4* __restrict__ units, const int64_t* __restrict__ offs,
                                                     int64_t nch, uint32_t* __restrict__ lc) {
    const int64_t i = offs[0] + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= offs[nch]) return;
    int64_t lo = 0, hi = nch - 1;  // the last chunk k with offs[k] <= i
    while (lo < hi) {
        const int64_t mid = (lo + hi + 1) >> 1;
        if (offs[mid] <= i) lo = mid;
        else hi = mid - 1;
    }
    atomicMax(&lc[units[i].z], (uint32_t)lo);
}

// off[k] = the first position of chunk number k in the ascending key[0, n)
// (n >= 1), off[nch] = n
__global__ __launch_bounds__(256) void k_chunk_starts(const uint32_t* __restrict__ key, int64_t n, int64_t nch,
                                                      int64_t* __restrict__ off) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int64_t k = key[i];
    const int64_t prev = i == 0 ? -1 : (int64_t)key[i - 1];
    for (int64_t j = prev + 1; j <= k; j++) off[j] = i;
    if (i == n - 1)
        for (int64_t j = k + 1; j <= nch; j++) off[j] = n;
}

// ------------------------------------------------------------- chunk index --

// The structures a layer streams over, fixed by (graph, chunk size, edge
// mask): the item sources grouped by (chunk, destination), per-vertex
// message counts |M(v)|, and per chunk the slices of the work lists.
// Exact layers over one graph and chunk size share one index.
struct ChunkIndex {
    Arena arena;
    taurus_graph g{};
    int64_t C = 0, nchunks = 0, kept = 0, segments = 0, max_long_per_chunk = 0;
    int64_t n_list[NLIST] = {};
    bool sampled = false;
    hipStream_t built_on = nullptr;
    hipEvent_t ready = nullptr;    // recorded after the last kernel that writes the index
    int32_t* m = nullptr;          // |M(v)|
    uint8_t* has_own = nullptr;    // per vertex: OWN_SEGMENT, SELF_FIRST
    unsigned long long* own_count = nullptr;  // number of such vertices
    int32_t* item_src = nullptr;   // local source row per item
    int4* units = nullptr;         // the work lists, one after another
    std::vector<int64_t> chunk_off;              // items before each chunk
    std::vector<int64_t> list_off[NLIST];        // buffer position of each chunk's first entry of list l
    double ms_build = 0;
    ChunkIndex(hipStream_t s, int64_t budget) : arena(s, budget), built_on(s) {}
    // The index may outlive the stream it was built on and be read from other
    // streams: wait for the device, then return the memory on the null stream.
    ~ChunkIndex() {
        (void)hipDeviceSynchronize();
        if (ready) (void)hipEventDestroy(ready);
        arena.set_stream(nullptr);
        arena.release();
    }
    const int4* list_at(int l, int64_t k) const { return units + list_off[l][(size_t)k]; }
    int64_t list_count(int l, int64_t k) const {
        return list_off[l][(size_t)k + 1] - list_off[l][(size_t)k];
    }
    // make stream s wait until the index is complete
    void wait_ready(hipStream_t s) const {
        if (ready && s != built_on) TAURUS_HIP(hipStreamWaitEvent(s, ready, 0));
    }
};

static void check_graph_args(const taurus_graph* g) {
    if (!g) fail(TAURUS_E_INVALID, "null graph");
    if (g->n <= 0 || g->n >= ((int64_t)1 << 31) || g->e < 0)
        fail(TAURUS_E_INVALID, "graph size n=%lld e=%lld out of range", (long long)g->n, (long long)g->e);
    if (!g->row_off || (g->e > 0 && !g->col_dst)) fail(TAURUS_E_INVALID, "graph arrays are null");
}

static double ms_since(std::chrono::steady_clock::time_point t0) {
    return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
}

// A sampled layer's index (sample != null) takes its items straight from the
// fanout sampler; an exact layer's from every CSR edge.
struct SampleReq {
    const Csc* csc;
    uint64_t seed;
    int layer, k;
};

// scratch (optional): where the build's temporaries go
static std::shared_ptr<ChunkIndex> build_index(const taurus_graph& g, int64_t C, const SampleReq* sample,
                                               hipStream_t s, int64_t budget, Arena* scratch = nullptr) {
    const auto t_start = std::chrono::steady_clock::now();
    auto idx = std::make_shared<ChunkIndex>(s, budget);
    const int64_t n = g.n, e = g.e;
    idx->g = g;
    idx->C = C;
    idx->nchunks = ceil_div(n, C);
    idx->sampled = sample != nullptr;
    const int T = 256;
    const int64_t nch = idx->nchunks;
    Arena own(s);
    Arena& tmp = scratch ? *scratch : own;
    auto finish = [&]() {
        TAURUS_HIP(hipEventCreateWithFlags(&idx->ready, hipEventDisableTiming));
        TAURUS_HIP(hipEventRecord(idx->ready, s));
        idx->ms_build = ms_since(t_start);
    };

    idx->m = idx->arena.alloc<int32_t>(n, "message counts");
    fill_i32(idx->m, n, 0, s);
    // a vertex without messages is SELF_FIRST; the flags of the others are
    // set once the segments are known
    idx->has_own = idx->arena.alloc<uint8_t>(ceil_div(n, 4) * 4, "per-vertex self-message flags");
    static_assert(SELF_FIRST == 2, "flag bytes are filled as 0x02");
    fill_i32(reinterpret_cast<int32_t*>(idx->has_own), ceil_div(n, 4), 0x02020202, s);
    idx->own_count = idx->arena.alloc<unsigned long long>(1, "own-chunk segment count");
    fill_i32(reinterpret_cast<int32_t*>(idx->own_count), 2, 0, s);
    idx->chunk_off.assign((size_t)nch + 1, 0);
    for (int l = 0; l < NLIST; l++) idx->list_off[l].assign((size_t)nch + 1, 0);
    // flags: 1, 2 invalid CSR; 4 unsorted row or self loop; 8 sort inconsistency
    int* bad = tmp.alloc<int>(1, "graph flag");
    fill_i32(bad, 1, 0, s);
    if (!sample) {  // a sampled layer's in-edge lists were built from a validated CSR
        k_validate_graph<<<(unsigned)ceil_div(std::max(n, e), T), T, 0, s>>>(g.row_off, g.col_dst, n, e, bad);
        TAURUS_CHECK_LAUNCH();
    }
    int hbad = 0;
    if (e == 0) {  // no messages: the self passes do all the work
        Readback rb;
        rb.add(&hbad, bad, 1);
        rb.run(s);
        if (hbad) fail(TAURUS_E_INVALID, "graph is not a valid CSR over [0, n) (flags %d)", hbad);
        finish();
        return idx;
    }

    // Items sorted by (source chunk, destination), stably.  Everything up to
    // the readback below is memory safe on an invalid graph (indices come
    // from binary searches and thread ids only); the flags are checked before
    // any kernel indexes by destination.
    const int vbits = std::max(1, bits_for(n - 1));
    const int cbits = bits_for(nch - 1);  // chunk numbers 0 .. nch - 1
    // the sampler's keys carry the not-first-flush bit between the fields
    const int kshift = sample ? vbits + 1 : vbits;
    if (kshift + cbits > 64) fail(TAURUS_E_INVALID, "index key does not fit 64 bits");
    SortBuffers sb{{nullptr, nullptr}, {nullptr, nullptr}, 0};
    int64_t items = e;
    int32_t* first_chunk = tmp.alloc<int32_t>(n, "first chunk per vertex");
    fill_i32(first_chunk, n, 0x7fffffff, s);
    if (sample) {
        // the sampler's kept in-edges come destination-major with sources
        // ascending, so a stable sort by the chunk field alone orders them
        // by (chunk, destination, source)
        items = sample_items(*sample->csc, n, sample->seed, sample->layer, sample->k, C, vbits, tmp, idx->arena, sb,
                             idx->m, first_chunk, bad, s);
        radix_sort_u64(sb, items, cbits, tmp, s, bad, 8, nullptr, kshift);
    } else {
        sb.keys[0] = tmp.alloc<uint64_t>(e, "index keys");
        sb.keys[1] = tmp.alloc<uint64_t>(e, "index keys (ping-pong)");
        // the sorted values become the index's item sources
        sb.vals[0] = idx->arena.alloc<uint32_t>(e, "index values");
        sb.vals[1] = idx->arena.alloc<uint32_t>(e, "index values (ping-pong)");
        k_make_items<<<(unsigned)ceil_div(e, MI_TILE), 256, 0, s>>>(g.row_off, g.col_dst, e, n, C, vbits,
                                                                    sb.keys[0], sb.vals[0], bad);
        TAURUS_CHECK_LAUNCH();
        radix_sort_u64(sb, items, vbits + cbits, tmp, s, bad, 8);
    }
    const int64_t items1 = std::max<int64_t>(items, 1);
    const uint64_t* keys = sb.keys[sb.cur];
    uint32_t* vals = sb.vals[sb.cur];
    tmp.free_ptr(sb.keys[1 - sb.cur]);
    idx->arena.free_ptr(sb.vals[1 - sb.cur]);
    int64_t* doffs = tmp.alloc<int64_t>(nch + 1, "chunk offsets");
    k_chunk_bounds<<<(unsigned)ceil_div(nch + 1, T), T, 0, s>>>(keys, items, nch, kshift, doffs);
    TAURUS_CHECK_LAUNCH();
    const int64_t nbt = ceil_div(items1, HEAD_TILE);
    uint64_t* hcount = tmp.alloc<uint64_t>(nbt, "segment heads per tile");
    uint64_t* hoff = tmp.alloc<uint64_t>(nbt + 1, "segment heads before each tile");
    k_head_counts<<<(unsigned)nbt, 256, 0, s>>>(keys, doffs + nch, hcount);
    TAURUS_CHECK_LAUNCH();
    scan_u64(hcount, hoff, nbt, true, tmp, s);
    uint64_t heads = 0;
    {
        Readback rb;
        rb.add(&hbad, bad, 1);
        rb.add(idx->chunk_off.data(), doffs, nch + 1);
        rb.add(&heads, hoff + nbt, 1);
        rb.run(s);
    }
    const int64_t P = (int64_t)heads;
    if (hbad & 3) fail(TAURUS_E_INVALID, "graph is not a valid CSR over [0, n) (flags %d)", hbad);
    if (hbad & 4) fail(TAURUS_E_INVALID, "graph rows are not strictly ascending or hold a self loop");
    if (hbad & 8) fail(TAURUS_E_DEVICE, "chunk index: radix sort offset out of range");
    if (hbad & 32) fail(TAURUS_E_INVALID, "sampler: an in-list holds repeated sources");
    const int64_t kept = idx->chunk_off[(size_t)nch];
    idx->kept = kept;
    idx->segments = P;
    if (kept == 0) {
        finish();
        return idx;
    }

    // segments into the work lists, list by list with one count buffer and
    // one offset buffer (two for the wave pieces and their fix-up entries)
    int64_t* seg_start = tmp.alloc<int64_t>(P + 1, "segment starts");
    k_head_positions<<<(unsigned)nbt, 256, 0, s>>>(keys, items, doffs + nch, hoff, P, seg_start);
    TAURUS_CHECK_LAUNCH();
    tmp.free_ptr(hoff);
    tmp.free_ptr(hcount);
    int32_t* slots_of = tmp.alloc<int32_t>(P, "segment slots");
    if (sample)
        k_seg_classify<true><<<(unsigned)ceil_div(P, T), T, 0, s>>>(keys, seg_start, P, vbits, kshift, C, idx->m,
                                                                    first_chunk, slots_of, idx->has_own,
                                                                    idx->own_count);
    else
        k_seg_classify<false><<<(unsigned)ceil_div(P, T), T, 0, s>>>(keys, seg_start, P, vbits, kshift, C, idx->m,
                                                                     first_chunk, slots_of, idx->has_own,
                                                                     idx->own_count);
    TAURUS_CHECK_LAUNCH();
    k_self_first<<<(unsigned)ceil_div(n, T), T, 0, s>>>(first_chunk, n, C, idx->has_own);
    TAURUS_CHECK_LAUNCH();
    // Unit positions: per tile of LT_TILE segments, the entries each list
    // takes (one pass), an exclusive scan over all lists' tiles one list
    // after another (the lists' buffer positions), then each tile writes its
    // units and its chunks' first positions (a second pass).
    const int64_t ntiles = ceil_div(P, LT_TILE);
    uint64_t* tile_cnt = tmp.alloc<uint64_t>(ntiles * NLIST, "list entries per tile");
    uint64_t* tile_off = tmp.alloc<uint64_t>(ntiles * NLIST + 1, "list positions per tile");
    k_list_tile_counts<<<(unsigned)ntiles, LT_THREADS, 0, s>>>(slots_of, P, ntiles, tile_cnt);
    TAURUS_CHECK_LAUNCH();
    scan_u64(tile_cnt, tile_off, ntiles * NLIST, true, tmp, s);
    int64_t list_base[NLIST + 1] = {0};
    {
        uint64_t lb[NLIST + 1] = {};
        Readback rb;
        for (int l = 0; l < NLIST; l++) rb.add(&lb[l], tile_off + (int64_t)l * ntiles, 1);
        rb.add(&lb[NLIST], tile_off + ntiles * NLIST, 1);
        rb.run(s);
        for (int l = 0; l <= NLIST; l++) list_base[l] = (int64_t)lb[l];
    }
    const int64_t total_units = list_base[NLIST];
    if (total_units >= ((int64_t)1 << 31)) fail(TAURUS_E_INVALID, "too many work units");
    idx->units = idx->arena.alloc<int4>(std::max<int64_t>(1, total_units), "work lists");
    int64_t* dbases = tmp.alloc<int64_t>((nch + 1) * NLIST, "chunk list positions");
    k_list_emit<<<(unsigned)ntiles, LT_THREADS, 0, s>>>(keys, seg_start, slots_of, P, ntiles, tile_off, vbits,
                                                       kshift, C, doffs, first_chunk, nch, idx->units, dbases);
    TAURUS_CHECK_LAUNCH();
    {
        std::vector<int64_t> bases((size_t)(nch + 1) * NLIST);
        Readback rb;
        rb.add(bases.data(), dbases, (nch + 1) * NLIST);
        rb.run(s);
        for (int l = 0; l < NLIST; l++) {
            for (int64_t k = 0; k <= nch; k++) idx->list_off[l][(size_t)k] = bases[(size_t)l * (nch + 1) + (size_t)k];
            idx->n_list[l] = list_base[l + 1] - list_base[l];
        }
    }
    for (int64_t k = 0; k < nch; k++)
        idx->max_long_per_chunk = std::max(idx->max_long_per_chunk, idx->list_count(NCLASS, k));
    idx->item_src = reinterpret_cast<int32_t*>(vals);  // local source rows, below C < 2^31
    finish();
    return idx;
}

}  // namespace taurus

namespace taurus {

// ------------------------------------------------------------------- GAT --
// Single-head GATConv (Sec. 3.9, GATConv) in three passes over the chunks:
//   1. transform (taurus_push_chunk): h'_c = X_c W for the chunk, written to
//      a table h' of every vertex, and two more columns s_u = a_src . h'_u
//      and t_u = a_dst . h'_u, taken in fp32 from the transformed row;
//   2. softmax statistics, topology only: per destination the largest score
//      m_v and the sum S_v = sum_u exp(e_uv - m_v) over its neighbourhood
//      (propagated messages and the self message), e_uv = LeakyReLU(s_u +
//      t_v).  Walks the chunk index in chunk order; each segment merges its
//      own (max, sum) into the destination's as the sole owner, hub pieces
//      through per-piece scalar carries merged in piece order, so the
//      result is deterministic;
//   3. aggregation: the chunks of h' are streamed again through the
//      scatter kernel of the other families (k_scatter<G, VEC, true>): every
//      message adds alpha_uv h'_u with alpha_uv = exp(e_uv - m_v) / S_v,
//      then the sole-owner flush and fix-up.
constexpr float GAT_SLOPE = ATT_SLOPE;

struct GatParams {
    const float* hp;  // [n][ystride]: h' then s, t
    int64_t ystride;
    int d_o;
    float* m;         // [n] running largest score
    float* S;         // [n] running sum of exp(score - m); 0 = none yet
    float* scarry;    // per hub piece of the chunk: {max, sum}
};

// pass 1 after the chunk's transform: one wave per row of h' (row stride
// ncols) writes s and t into columns d_o and d_o + 1
__global__ __launch_bounds__(256) void k_gat_scores(float* __restrict__ hp, int64_t rows, int64_t ncols, int d_o,
                                                    const float* __restrict__ attn) {
    const int lane = threadIdx.x & 63;
    const int64_t r = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (r >= rows) return;
    float* row = hp + r * ncols;
    float s = 0.f, t = 0.f;
    for (int o = lane; o < d_o; o += 64) {
        s = fmaf(attn[o], row[o], s);
        t = fmaf(attn[d_o + o], row[o], t);
    }
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) {
        s += __shfl_xor(s, d, 64);
        t += __shfl_xor(t, d, 64);
    }
    if (lane == 0) {
        row[d_o] = s;
        row[d_o + 1] = t;
    }
}

__device__ inline float gat_score(const GatParams& q, int64_t u, int64_t v) {
    const float e = q.hp[u * q.ystride + q.d_o] + q.hp[v * q.ystride + q.d_o + 1];
    return e > 0.f ? e : GAT_SLOPE * e;
}

// (m, S) <- the statistics of both parts
__device__ inline void gat_merge(float& m, float& S, float m2, float S2) {
    if (S2 == 0.f) return;
    if (S == 0.f) {
        m = m2;
        S = S2;
        return;
    }
    const float M = fmaxf(m, m2);
    S = S * expf(m - M) + S2 * expf(m2 - M);
    m = M;
}

// Source vertex of slot i of a short unit (slot 0 of a SELF_HERE unit is
// the destination itself) or of a wave piece (its last slot, with
// SELF_HERE).
__device__ inline int64_t short_slot_src(const ScatterParams& p, int4 w, int i) {
    const int self = (w.y & SELF_HERE) ? 1 : 0;
    return (self && i == 0) ? (int64_t)w.z : p.first_row + p.src[w.x + i - self];
}
__device__ inline int64_t piece_slot_src(const ScatterParams& p, int4 w, int i) {
    const int items = (w.y & LEN_MASK) - ((w.y & SELF_HERE) ? 1 : 0);
    return i < items ? p.first_row + p.src[w.x + i] : (int64_t)w.z;
}

// unit t of the chunk's short classes taken as one sequence
__device__ inline int4 short_unit(const ChunkUnits& cu, int64_t t) {
#pragma unroll
    for (int c = 0; c < NCLASS; c++) {
        if (t < cu.n[c]) return cu.u[c][t];
        t -= cu.n[c];
    }
    return make_int4(0, 0, -1, 0);
}

// pass 2, short units: one thread each
__global__ void k_gat_stats_short(ScatterParams p, ChunkUnits cu, GatParams q, int64_t total) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= total) return;
    const int4 w = short_unit(cu, t);
    const int v = w.z, L = w.y & LEN_MASK;
    float mx = -INFINITY;
    for (int i = 0; i < L; i++) mx = fmaxf(mx, gat_score(q, short_slot_src(p, w, i), v));
    float sum = 0.f;
    for (int i = 0; i < L; i++) sum += expf(gat_score(q, short_slot_src(p, w, i), v) - mx);
    float m = q.m[v], S = q.S[v];
    gat_merge(m, S, mx, sum);
    q.m[v] = m;
    q.S[v] = S;
}

// pass 2, wave pieces: one wave each; a hub piece parks its statistics
__global__ __launch_bounds__(256) void k_gat_stats_pieces(ScatterParams p, const int4* __restrict__ units,
                                                          int64_t n, GatParams q) {
    const int lane = threadIdx.x & 63;
    const int64_t un = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (un >= n) return;  // the whole wave
    const int4 w = units[un];
    const int v = w.z, L = w.y & LEN_MASK;
    float mx = -INFINITY;
    for (int i = lane; i < L; i += 64) mx = fmaxf(mx, gat_score(q, piece_slot_src(p, w, i), v));
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) mx = fmaxf(mx, __shfl_xor(mx, d, 64));
    float sum = 0.f;
    for (int i = lane; i < L; i += 64) sum += expf(gat_score(q, piece_slot_src(p, w, i), v) - mx);
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) sum += __shfl_xor(sum, d, 64);
    if (lane != 0) return;
    if (w.w < 0) {
        float m = q.m[v], S = q.S[v];
        gat_merge(m, S, mx, sum);
        q.m[v] = m;
        q.S[v] = S;
    } else {
        const int64_t slot = (int64_t)w.w - p.long_base;
        q.scarry[2 * slot] = mx;
        q.scarry[2 * slot + 1] = sum;
    }
}

// pass 2, the chunk's own vertices without a segment from it, and the hub
// segments' pieces in order
__global__ void k_gat_stats_self(ScatterParams p, GatParams q) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= p.rows) return;
    const int64_t v = p.first_row + r;
    if (p.has_own[v] & OWN_SEGMENT) return;
    float m = q.m[v], S = q.S[v];
    gat_merge(m, S, gat_score(q, v, v), 1.f);
    q.m[v] = m;
    q.S[v] = S;
}
__global__ void k_gat_stats_fixup(ScatterParams p, const int4* __restrict__ fix, int64_t nfix, GatParams q) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= nfix) return;
    const int4 f = fix[t];
    const int v = f.x;
    const int64_t first = (int64_t)f.y - p.long_base;
    float m = q.m[v], S = q.S[v];
    for (int j = 0; j < f.z; j++) gat_merge(m, S, q.scarry[2 * (first + j)], q.scarry[2 * (first + j) + 1]);
    q.m[v] = m;
    q.S[v] = S;
}

}  // namespace taurus

// ------------------------------------------------------------- handles -----

struct taurus_plan {
    taurus_graph g{};
    int64_t chunk = 0;
    // built by the first layer that needs them, on that layer's stream
    std::mutex mu;
    std::shared_ptr<taurus::ChunkIndex> idx;  // exact layers
    std::shared_ptr<taurus::Csc> csc;         // sampled layers
    double ms_build = 0;                      // time the plan's structures took to build
};

struct taurus_layer {
    taurus_graph g{};
    taurus_layer_desc d{};
    hipStream_t s = nullptr;
    taurus::Arena arena;
    std::shared_ptr<taurus::ChunkIndex> idx;
    bool poisoned = false;
    int64_t n = 0, C = 0, nchunks = 0;
    int d_o = 0, ncols = 0;
    int ystride = 0;  // row stride of the chunk transform Y (floats)
    taurus::ScatterShape shape{};
    int2* cnt = nullptr;
    float* n_out = nullptr;
    float* acc = nullptr;
    float* wpack = nullptr;
    float* bias = nullptr;
    float* Y = nullptr;
    float* carry = nullptr;
    int32_t* carry_cnt = nullptr;
    // in-core fp32 GCN and linear-apply GIN layers run the fix-up of chunk j
    // inside the transform launch of the next chunk pushed (or at finalize)
    bool fuse_fix = false, fix_pending = false;
    // in-core GraphSAGE layers: each chunk's transform takes the self
    // messages of the vertices without a segment from their own chunk
    // (SelfFlush), so those rows' self halves never pass through Y
    bool self_in_transform = false;
    unsigned long long* self_tally = nullptr;  // profiled layers: [TALLY_SLOTS][2]
    taurus::ScatterParams fix_p{};
    const int4* fix_list = nullptr;
    int64_t fix_n = 0;
    uint64_t* mask = nullptr;    // sampled layers: CSR-order mask, drawn when first needed
    std::shared_ptr<taurus::Csc> csc;  // sampled layers: the in-edge lists the sample is drawn from
    float* gat_hp = nullptr;     // GAT: h' of every vertex, then s, t ([n][ncols])
    float* gat_m = nullptr;      // GAT: per-destination largest score
    float* gat_s = nullptr;      // GAT: per-destination sum of exp(score - max)
    float* gat_carry = nullptr;  // GAT: per hub piece {max, sum}
    const float* gat_attn = nullptr;  // GAT: a_src then a_dst on the device
    bool gat_done = false;       // GAT: passes 2 and 3 have run
    bool acc_deferred = false;   // dense accumulators allocated by the first push
    // GIN with a perceptron: the second layer (packed for the matrix cores)
    // and its bias; the destinations grouped by the chunk they complete in
    // (comp_ids), chunk k's at [comp_off[k], comp_off[k + 1])
    float* w2pack = nullptr;
    float* bias2 = nullptr;
    int32_t* comp_ids = nullptr;
    std::vector<int64_t> comp_off;
    int grad_blocks = 0;
    void* wpack_any = nullptr;  // packed weights (fp32 or 16-bit fragments)
    void* out_dev = nullptr;    // desc.out as kernels address it
    std::unique_ptr<taurus::Residency> res;  // accumulator pool under a budget (null: dense rows)
    // host-resident chunks: two device staging buffers filled on a copy stream
    hipStream_t copy_stream = nullptr;
    void* stage[2] = {nullptr, nullptr};
    hipEvent_t h2d_done[2] = {nullptr, nullptr}, gemm_done[2] = {nullptr, nullptr};
    bool stage_used[2] = {false, false};
    int64_t host_pushes = 0, h2d_bytes = 0;
    std::vector<uint8_t> pushed;
    int64_t npushed = 0;
    double ms_init = 0, ms_index = 0;
    std::vector<hipEvent_t> events;  // EV_PER_CHUNK per chunk when profiling
    ~taurus_layer();
};

namespace taurus {

// events per pushed chunk: before the transform, the scatter (self pass
// included), the fix-up, and after it
constexpr int EV_PER_CHUNK = 4;

// Timing events are recycled across layers (creating them costs more than
// recording them).
static std::mutex g_event_mu;
static std::vector<hipEvent_t>* g_free_events = new std::vector<hipEvent_t>();

static hipEvent_t timing_event_acquire() {
    {
        std::lock_guard<std::mutex> g(g_event_mu);
        if (!g_free_events->empty()) {
            hipEvent_t ev = g_free_events->back();
            g_free_events->pop_back();
            return ev;
        }
    }
    hipEvent_t ev = nullptr;
    TAURUS_HIP(hipEventCreate(&ev));
    return ev;
}

static void timing_event_release(hipEvent_t ev) {
    if (!ev) return;
    std::lock_guard<std::mutex> g(g_event_mu);
    g_free_events->push_back(ev);
}

}  // namespace taurus

taurus_layer::~taurus_layer() {
    for (auto ev : events) taurus::timing_event_release(ev);
    if (copy_stream) {
        (void)hipStreamSynchronize(copy_stream);
        for (int i = 0; i < 2; i++) {
            if (h2d_done[i]) (void)hipEventDestroy(h2d_done[i]);
            if (gemm_done[i]) (void)hipEventDestroy(gemm_done[i]);
        }
        (void)hipStreamDestroy(copy_stream);
    }
}

namespace taurus {

// Graduation lists of a GIN layer with a perceptron: the vertices grouped
// (stably) by the chunk they complete in, built once from the chunk index,
// so that a push knows the rows it hands to W2 without the scatter keeping
// a list.  Temporaries come from tmp.
static void build_completion_lists(taurus_layer* L, const ChunkIndex& idx, Arena& tmp, hipStream_t s) {
    const int T = 256;
    const int64_t n = L->n, nch = L->nchunks;
    SortBuffers32 sb{{tmp.alloc<uint32_t>(n, "completing chunks"), tmp.alloc<uint32_t>(n, "completing chunks (ping-pong)")},
                     {tmp.alloc<uint32_t>(n, "completing vertices"),
                      tmp.alloc<uint32_t>(n, "completing vertices (ping-pong)")},
                     0};
    k_own_chunk<<<(unsigned)ceil_div(n, T), T, 0, s>>>(sb.keys[0], sb.vals[0], n, L->C);
    TAURUS_CHECK_LAUNCH();
    // the short classes' and the wave units' positions per chunk (the
    // fix-up list names hubs that the wave units name too)
    constexpr int NL = NCLASS + 1;
    const size_t obytes = (size_t)NL * (size_t)(nch + 1) * sizeof(int64_t);
    int64_t* stage = static_cast<int64_t*>(pinned_staging(obytes));
    for (int l = 0; l < NL; l++)
        for (int64_t k = 0; k <= nch; k++) stage[(size_t)l * (nch + 1) + (size_t)k] = idx.list_off[l][(size_t)k];
    int64_t* offs = tmp.alloc<int64_t>((int64_t)NL * (nch + 1), "work-list positions");
    TAURUS_HIP(hipMemcpyAsync(offs, stage, obytes, hipMemcpyHostToDevice, s));
    pinned_staging_in_flight(s);
    for (int l = 0; l < NL; l++) {
        const int64_t cnt = idx.list_off[l][(size_t)nch] - idx.list_off[l][0];
        if (cnt <= 0) continue;
        k_unit_chunks<<<(unsigned)ceil_div(cnt, T), T, 0, s>>>(idx.units, offs + (int64_t)l * (nch + 1), nch,
                                                               sb.keys[0]);
        TAURUS_CHECK_LAUNCH();
    }
    int* bad = tmp.alloc<int>(1, "sort flag");
    fill_i32(bad, 1, 0, s);
    radix_sort_u32(sb, n, std::max(1, bits_for(nch - 1)), tmp, s, bad, 0);
    int64_t* off = tmp.alloc<int64_t>(nch + 1, "graduation list positions");
    k_chunk_starts<<<(unsigned)ceil_div(n, T), T, 0, s>>>(sb.keys[sb.cur], n, nch, off);
    TAURUS_CHECK_LAUNCH();
    L->comp_ids = L->arena.alloc<int32_t>(n, "graduation lists");
    TAURUS_HIP(hipMemcpyAsync(L->comp_ids, sb.vals[sb.cur], (size_t)n * 4, hipMemcpyDeviceToDevice, s));
    L->comp_off.assign((size_t)nch + 1, 0);
    int hbad = 0;
    Readback rb;
    rb.add(L->comp_off.data(), off, nch + 1);
    rb.add(&hbad, bad, 1);
    rb.run(s);
    if (hbad || L->comp_off[0] != 0 || L->comp_off[(size_t)nch] != n)
        fail(TAURUS_E_DEVICE, "graduation lists are inconsistent (flags %d)", hbad);
}

static void validate_desc(const taurus_layer_desc* d) {
    if (!d) fail(TAURUS_E_INVALID, "null descriptor");
    if (d->agg != TAURUS_SAGE_MEAN && d->agg != TAURUS_GCN_SYM && d->agg != TAURUS_GIN_SUM &&
        d->agg != TAURUS_GAT_ATT && d->agg != TAURUS_GIN_MLP)
        fail(TAURUS_E_INVALID, "unknown agg %d", d->agg);
    if (d->agg == TAURUS_GIN_MLP) {
        if (d->d_hidden <= 0 || d->d_hidden % 4 || d->d_hidden > 1024)
            fail(TAURUS_E_INVALID, "d_hidden=%d: a positive multiple of 4, at most 1024", d->d_hidden);
        if (!d->weight2) fail(TAURUS_E_INVALID, "a GIN perceptron layer needs weight2");
        if (d->hbm_budget != 0) fail(TAURUS_E_INVALID, "GIN perceptron layers run in core (hbm_budget 0)");
    }
    if (d->agg == TAURUS_GAT_ATT && !d->attn) fail(TAURUS_E_INVALID, "a GAT layer needs its attention vectors");
    if (d->agg == TAURUS_GAT_ATT && d->hbm_budget != 0)
        fail(TAURUS_E_INVALID, "GAT layers run in core (hbm_budget must be 0)");
    if (d->d_in <= 0 || d->d_out <= 0 || d->d_in % 4 || d->d_out % 4 || d->d_out > 1024 || d->d_in > 8192)
        fail(TAURUS_E_INVALID, "d_in=%d d_out=%d: widths must be positive multiples of 4, d_out <= 1024",
             d->d_in, d->d_out);
    if (d->in_dtype < TAURUS_F32 || d->in_dtype > TAURUS_F16) fail(TAURUS_E_INVALID, "in_dtype %d", d->in_dtype);
    if (d->in_dtype != TAURUS_F32 && d->d_in % 8)
        fail(TAURUS_E_INVALID, "d_in=%d: 16-bit inputs need a multiple of 8", d->d_in);
    if (d->out_dtype < 0 || d->out_dtype > 2) fail(TAURUS_E_INVALID, "out_dtype %d", d->out_dtype);
    if (!d->weight) fail(TAURUS_E_INVALID, "weight is null");
    if (d->chunk <= 0 || d->chunk >= ((int64_t)1 << 31)) fail(TAURUS_E_INVALID, "chunk %lld", (long long)d->chunk);
    if (d->fanout < 0 || d->fanout > FANOUT_MAX)
        fail(TAURUS_E_INVALID, "fanout %d outside [0, %d]", d->fanout, FANOUT_MAX);
    if (d->fanout > 0 && d->layer < 1) fail(TAURUS_E_INVALID, "layer %d: sampled layers are numbered from 1", d->layer);
    if (!d->out) fail(TAURUS_E_INVALID, "out is null");
    if (d->out_on_host != 0 && d->out_on_host != 1) fail(TAURUS_E_INVALID, "out_on_host=%d", d->out_on_host);
    if (d->hub_fraction < 0.0 || d->hub_fraction > 1.0) fail(TAURUS_E_INVALID, "hub_fraction %g", d->hub_fraction);
    if (d->eviction < TAURUS_EVICT_PENDING || d->eviction > TAURUS_EVICT_LRU)
        fail(TAURUS_E_INVALID, "eviction policy %d", (int)d->eviction);
    if (d->hbm_budget < 0) fail(TAURUS_E_INVALID, "hbm_budget < 0");
    if (d->profile < 0 || d->profile > 2) fail(TAURUS_E_INVALID, "profile %d", d->profile);
}

static bool same_graph(const taurus_graph& a, const taurus_graph& b) {
    return a.n == b.n && a.e == b.e && a.row_off == b.row_off && a.col_dst == b.col_dst;
}

static void layer_init(taurus_layer* L) {
    const auto t_start = std::chrono::steady_clock::now();
    // the set-up work goes to desc.setup_stream when given (the layer's
    // stream waits for it at the end), else to the layer's stream
    hipStream_t s = L->d.setup_stream ? static_cast<hipStream_t>(L->d.setup_stream) : L->s;
    L->arena.set_stream(s);
    const taurus_graph& g = L->g;
    const taurus_layer_desc& d = L->d;
    const int64_t n = g.n, C = d.chunk;
    L->n = n;
    L->C = C;
    L->nchunks = ceil_div(n, C);
    // accumulator width: the perceptron's hidden width for GIN_MLP
    L->d_o = d.agg == TAURUS_GIN_MLP ? d.d_hidden : d.d_out;
    // GraphSAGE: [W_agg | W_self]; GAT: W and the two attention columns,
    // padded to a multiple of 4
    L->ncols = d.agg == TAURUS_SAGE_MEAN ? 2 * d.d_out : d.agg == TAURUS_GAT_ATT ? d.d_out + 4 : L->d_o;
    // Y rows padded to whole 128-byte lines (the padding columns hold the
    // zero-padded weights' products): the transform then writes whole lines
    // and a gathered row starts on a line
    L->ystride = d.agg == TAURUS_GAT_ATT ? L->ncols : (L->ncols + 31) / 32 * 32;
    L->shape = scatter_shape(L->d_o);
    L->shape.max_blocks = scatter_resident_blocks(L->shape, false);
    L->shape.max_blocks_att = scatter_resident_blocks(L->shape, true);
    const int T = 256;

    // chunk index: exact layers share the plan's (built here if it is the
    // first user); a sampled layer draws its mask (from the plan's CSC) and
    // builds its own index of the kept edges
    taurus_plan* plan = const_cast<taurus_plan*>(d.plan);
    if (plan && (!same_graph(plan->g, g) || plan->chunk != C))
        fail(TAURUS_E_INVALID, "plan was built for another graph or chunk size");
    // Without a budget the accumulators are dense: they are allocated first
    // and, until the first chunk arrives (their rows are logically zero
    // while nothing has arrived and are never cleared), hold the temporaries
    // of the in-edge lists and the chunk index, so that those take no memory
    // of their own.
    // With a set-up stream the dense accumulators wait for the first push
    // instead (the layer before, whose chunks the set-up overlaps, may hold
    // its own until then), and the index takes memory of its own meanwhile.
    std::unique_ptr<Arena> scratch;
    const bool defer_acc = d.hbm_budget == 0 && s != L->s;
    if (d.hbm_budget == 0 && !defer_acc) {
        const int64_t acc_elems = n * (int64_t)L->d_o;
        L->acc = L->arena.alloc<float>(acc_elems, "accumulators");
        scratch = std::make_unique<Arena>(s, L->acc, acc_elems * 4, true);
    }
    const auto t_index = std::chrono::steady_clock::now();
    if (d.fanout > 0) {
        std::shared_ptr<Csc> csc;
        if (plan) {
            std::lock_guard<std::mutex> lock(plan->mu);
            if (!plan->csc) {
                plan->csc = build_csc(g, s, scratch.get());
                plan->ms_build += plan->csc->ms_build;
            }
            csc = plan->csc;
        } else {
            csc = build_csc(g, s, scratch.get());
        }
        if (scratch) scratch->release();
        const SampleReq req{csc.get(), d.seed, d.layer, d.fanout};
        L->idx = build_index(g, C, &req, s, 0, scratch.get());
        L->csc = csc;
        if (d.agg == TAURUS_GCN_SYM) {
            // the source norms count kept out-edges: the mask in CSR order
            L->mask = L->arena.alloc<uint64_t>(std::max<int64_t>(1, ceil_div(g.e, 64)), "fanout mask");
            sample_mask(g, *csc, d.seed, d.layer, d.fanout, L->mask, s);
        }
    } else if (plan) {
        std::lock_guard<std::mutex> lock(plan->mu);
        if (!plan->idx) {
            plan->idx = build_index(g, C, nullptr, s, 0, scratch.get());
            plan->ms_build += plan->idx->ms_build;
        }
        L->idx = plan->idx;
        L->idx->wait_ready(s);
    } else {
        L->idx = build_index(g, C, nullptr, s, 0, scratch.get());
    }
    if (scratch) scratch->release();
    L->ms_index = ms_since(t_index);
    const ChunkIndex& idx = *L->idx;

    L->cnt = L->arena.alloc<int2>(n, "pending counts");
    k_init_counts<<<(unsigned)ceil_div(n, T), T, 0, s>>>(idx.m, n, L->cnt);
    TAURUS_CHECK_LAUNCH();
    if (d.agg == TAURUS_GCN_SYM) {
        L->n_out = L->arena.alloc<float>(n, "source norms");
        if (L->mask) {
            // kept edges before each mask word (words + 1 entries: a row may
            // end at e, a multiple of 64)
            const int64_t words = std::max<int64_t>(1, ceil_div(g.e, 64));
            Arena tmp(s);
            uint32_t* wcnt = tmp.alloc<uint32_t>(words, "kept edges per mask word");
            uint64_t* woff = tmp.alloc<uint64_t>(words + 1, "kept edges before each mask word");
            k_mask_word_counts<<<(unsigned)ceil_div(words, T), T, 0, s>>>(L->mask, words, g.e, wcnt);
            TAURUS_CHECK_LAUNCH();
            scan_u32_to_u64(wcnt, woff, words, true, tmp, s);
            k_out_norm_kept<<<(unsigned)ceil_div(n, T), T, 0, s>>>(g.row_off, L->mask, woff, n, L->n_out);
        } else
            k_out_norm<<<(unsigned)ceil_div(n, T), T, 0, s>>>(g.row_off, n, L->n_out);
        TAURUS_CHECK_LAUNCH();
    }

    // packed weights and bias, one transfer through pinned staging (the
    // staging buffer's next user waits for it)
    std::vector<float> packed32;
    std::vector<uint16_t> packed16;
    size_t wbytes = 0;
    const float* wsrc = d.weight;
    std::vector<float> wext;
    if (d.agg == TAURUS_GAT_ATT) {
        // [W^T | 0 0 0 0]: the four extra columns of h' (the two attention
        // terms and padding) are filled after the transform
        wext.assign((size_t)d.d_in * L->ncols, 0.0f);
        for (int i = 0; i < d.d_in; i++)
            for (int o = 0; o < d.d_out; o++) wext[(size_t)i * L->ncols + o] = d.weight[(size_t)i * d.d_out + o];
        wsrc = wext.data();
    }
    if (d.in_dtype == TAURUS_F32) {
        gemm_pack_weights_f32(wsrc, d.d_in, L->ncols, packed32);
        wbytes = packed32.size() * 4;
    } else {
        gemm_pack_weights_16(wsrc, d.d_in, L->ncols, d.in_dtype, packed16);
        wbytes = packed16.size() * 2;
    }
    wbytes = (wbytes + 255) / 256 * 256;
    // bias, then (GAT) the attention vectors a_src, a_dst
    const int nattn = d.agg == TAURUS_GAT_ATT ? 2 * L->d_o : 0;
    // GIN with a perceptron: its second layer (fp32, packed) and bias after
    std::vector<float> packed2;
    if (d.agg == TAURUS_GIN_MLP) gemm_pack_weights_f32(d.weight2, d.d_hidden, d.d_out, packed2);
    const size_t w2off = (wbytes + (size_t)(L->d_o + nattn) * 4 + 255) / 256 * 256;
    const size_t pbytes = packed2.empty() ? wbytes + (size_t)(L->d_o + nattn) * 4
                                          : w2off + packed2.size() * 4 + (size_t)d.d_out * 4;
    char* stage = static_cast<char*>(pinned_staging(pbytes));
    if (!packed32.empty()) std::memcpy(stage, packed32.data(), packed32.size() * 4);
    if (!packed16.empty()) std::memcpy(stage, packed16.data(), packed16.size() * 2);
    float* sbias = reinterpret_cast<float*>(stage + wbytes);
    for (int j = 0; j < L->d_o; j++) sbias[j] = d.bias ? d.bias[j] : 0.0f;
    for (int j = 0; j < nattn; j++) sbias[L->d_o + j] = d.attn[j];
    if (!packed2.empty()) {
        std::memcpy(stage + w2off, packed2.data(), packed2.size() * 4);
        float* sb2 = reinterpret_cast<float*>(stage + w2off + packed2.size() * 4);
        for (int j = 0; j < d.d_out; j++) sb2[j] = d.bias2 ? d.bias2[j] : 0.0f;
    }
    L->wpack_any = L->arena.alloc_bytes((int64_t)pbytes, "packed weights and bias");
    L->wpack = static_cast<float*>(L->wpack_any);
    L->bias = reinterpret_cast<float*>(static_cast<char*>(L->wpack_any) + wbytes);
    if (nattn) L->gat_attn = L->bias + L->d_o;
    if (!packed2.empty()) {
        L->w2pack = reinterpret_cast<float*>(static_cast<char*>(L->wpack_any) + w2off);
        L->bias2 = L->w2pack + packed2.size();
    }
    TAURUS_HIP(hipMemcpyAsync(L->wpack_any, stage, pbytes, hipMemcpyHostToDevice, s));
    pinned_staging_in_flight(s);

    // output as kernels address it: device memory, or pinned host memory
    // mapped into the device's address space
    if (d.out_on_host) {
        if (hipHostGetDevicePointer(&L->out_dev, d.out, 0) != hipSuccess) {
            (void)hipGetLastError();
            fail(TAURUS_E_INVALID, "out_on_host = 1 but out is not pinned host memory");
        }
    } else {
        L->out_dev = d.out;
    }

    // working buffers
    // the scatter addresses Y with 32-bit byte offsets
    if (std::min<int64_t>(C, n) * (int64_t)L->ystride * 4 > (int64_t)0x7f000000)
        fail(TAURUS_E_INVALID, "chunk %lld x %d transform columns exceeds 2 GiB of fp32", (long long)C, L->ystride);
    if (d.agg == TAURUS_GAT_ATT) {
        L->gat_hp = L->arena.alloc<float>(n * (int64_t)L->ncols, "GAT transformed rows and scores");
        L->gat_m = L->arena.alloc<float>(n, "GAT largest scores");
        L->gat_s = L->arena.alloc<float>(n, "GAT score sums");
        fill_i32(reinterpret_cast<int32_t*>(L->gat_s), n, 0, s);
        L->gat_carry = L->arena.alloc<float>(2 * std::max<int64_t>(1, idx.max_long_per_chunk), "GAT piece statistics");
    } else {
        L->Y = L->arena.alloc<float>(std::min<int64_t>(C, n) * (int64_t)L->ystride, "chunk transform");
    }
    const int64_t carry_rows = std::max<int64_t>(1, idx.max_long_per_chunk);
    L->carry = L->arena.alloc<float>(carry_rows * L->d_o, "hub piece carries");
    L->carry_cnt = L->arena.alloc<int32_t>(carry_rows, "hub piece counts");
    L->pushed.assign((size_t)L->nchunks, 0);

    // Accumulators: dense rows [n][d_out] when they fit the budget; else a
    // pool of slots with resident hubs and eviction to pinned host memory.
    const int64_t row_bytes = (int64_t)L->d_o * 4;
    const int64_t index_bytes = L->idx->arena.bytes();
    const int64_t dense = n * row_bytes;
    if (L->acc) {
        // allocated before the index (no budget)
    } else if (defer_acc) {
        L->acc_deferred = true;
    } else if (L->arena.bytes() + index_bytes + dense + (dense >> 3) <= d.hbm_budget) {
        L->acc = L->arena.alloc<float>(n * (int64_t)L->d_o, "accumulators");
    } else {
        const int64_t staging = 2 * std::min(C, n) * (int64_t)d.d_in * (d.in_dtype == TAURUS_F32 ? 4 : 2) * 9 / 8;
        const int64_t avail =
            d.hbm_budget - L->arena.bytes() - index_bytes - Residency::fixed_bytes(n) * 9 / 8 - staging;
        const int64_t S = std::min<int64_t>(n, std::max<int64_t>(0, avail) * 8 / 9 / (row_bytes + 4));
        const int64_t H = (int64_t)std::ceil(d.hub_fraction * (double)n);
        int64_t max_dc = 0;
        for (int64_t k = 0; k < L->nchunks; k++) {
            int64_t t = std::min(C, n - k * C);
            for (int l = 0; l <= NCLASS; l++) t += idx.list_count(l, k);
            max_dc = std::max(max_dc, t);
        }
        if (S < H + std::min(max_dc, n - H))
            fail(TAURUS_E_BUDGET,
                 "budget %lld leaves %lld accumulator slots; %lld hubs plus one chunk's %lld destinations need more",
                 (long long)d.hbm_budget, (long long)S, (long long)H, (long long)max_dc);
        L->res = std::make_unique<Residency>(s, n, L->d_o, S, H, idx.m, idx.kept, d.eviction, d.seed, L->nchunks);
        const int64_t total = L->arena.bytes() + index_bytes + L->res->arena.bytes();
        if (total > d.hbm_budget)
            fail(TAURUS_E_BUDGET, "residency structures take %lld bytes, above the budget %lld", (long long)total,
                 (long long)d.hbm_budget);
    }
    if (d.agg == TAURUS_GIN_MLP) {
        // the accumulators are not in use yet: their memory holds the
        // temporaries here too
        Arena own(s);
        build_completion_lists(L, idx, scratch ? *scratch : own, s);
        if (scratch) scratch->release();
        int dev = 0, cus = 0;
        TAURUS_HIP(hipGetDevice(&dev));
        TAURUS_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
        L->grad_blocks = 2 * std::max(1, cus);   // at most two workgroups per compute unit
    }
    // the perceptron's graduation reads every flush of the chunk, the
    // fix-up's included, so its fix-up is not deferred
    // The transform of a chunk that takes self messages must not run beside
    // the previous chunk's fix-up, which may flush the same rows
    L->self_in_transform = d.agg == TAURUS_SAGE_MEAN && !L->res;
    L->fuse_fix = !L->res && !L->gat_hp && d.in_dtype == TAURUS_F32 && d.agg != TAURUS_GIN_MLP &&
                  !L->self_in_transform;
    if (L->self_in_transform && d.profile) {
        L->self_tally = L->arena.alloc<unsigned long long>(2 * TALLY_SLOTS, "self-message tallies");
        fill_i32(reinterpret_cast<int32_t*>(L->self_tally), 4 * TALLY_SLOTS, 0, s);
    }
    if (d.profile) {
        L->events.assign((size_t)L->nchunks * EV_PER_CHUNK, nullptr);
        for (auto& ev : L->events) ev = timing_event_acquire();
    }
    if (s != L->s) {
        // the layer's stream takes up the layer's memory and work from here
        hipEvent_t ready = nullptr;
        TAURUS_HIP(hipEventCreateWithFlags(&ready, hipEventDisableTiming));
        const hipError_t rc1 = hipEventRecord(ready, s);
        const hipError_t rc2 = rc1 == hipSuccess ? hipStreamWaitEvent(L->s, ready, 0) : rc1;
        (void)hipEventDestroy(ready);  // released once the wait has been satisfied
        TAURUS_HIP(rc2);
        L->arena.set_stream(L->s);
        if (L->res) L->res->arena.set_stream(L->s);
    }
    L->ms_init = ms_since(t_start);  // host time; the work stays queued on the stream
}

// Host-resident chunk (pinned): copy it on the layer's copy stream into one
// of two device staging buffers while the previous chunk computes.  A
// buffer is refilled only after the transform that read it; the caller's x
// must stay valid until the next call returns, so the previous chunk's copy
// is waited for here.
static const void* stage_host_chunk(taurus_layer* L, const void* x, int64_t rows) {
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, x) != hipSuccess || attr.type != hipMemoryTypeHost) {
        (void)hipGetLastError();
        fail(TAURUS_E_INVALID, "x_on_host = 1 but x is not pinned host memory");
    }
    const size_t elem = L->d.in_dtype == TAURUS_F32 ? 4 : 2;
    const size_t bytes = (size_t)rows * (size_t)L->d.d_in * elem;
    if (!L->copy_stream) {
        TAURUS_HIP(hipStreamCreateWithFlags(&L->copy_stream, hipStreamNonBlocking));
        for (int i = 0; i < 2; i++) {
            L->stage[i] = L->arena.alloc_bytes((int64_t)(std::min(L->C, L->n) * L->d.d_in * elem), "chunk staging");
            TAURUS_HIP(hipEventCreateWithFlags(&L->h2d_done[i], hipEventDisableTiming));
            TAURUS_HIP(hipEventCreateWithFlags(&L->gemm_done[i], hipEventDisableTiming));
        }
    }
    const int prev = (int)((L->host_pushes + 1) & 1), cur = (int)(L->host_pushes & 1);
    if (L->stage_used[cur]) TAURUS_HIP(hipStreamWaitEvent(L->copy_stream, L->gemm_done[cur], 0));
    TAURUS_HIP(hipMemcpyAsync(L->stage[cur], x, bytes, hipMemcpyHostToDevice, L->copy_stream));
    TAURUS_HIP(hipEventRecord(L->h2d_done[cur], L->copy_stream));
    TAURUS_HIP(hipStreamWaitEvent(L->s, L->h2d_done[cur], 0));
    // the previous chunk's x is released to the caller once its copy is done;
    // waiting after this chunk's copy is queued keeps the copy engine busy
    if (L->stage_used[prev]) TAURUS_HIP(hipEventSynchronize(L->h2d_done[prev]));
    L->stage_used[cur] = true;
    L->host_pushes++;
    L->h2d_bytes += (int64_t)bytes;
    return L->stage[cur];
}

// The fp32 transform of one chunk and the fix-up of the chunk pushed before
// it, in one launch: workgroups [0, gblocks) are the transform's row panels
// (gx per column group), the rest take the fix-up's hub segments.  Both only
// follow that earlier chunk's scatter on the stream, and this chunk's
// scatter follows both; one launch instead of two keeps the fix-up's few
// workgroups off the critical path.
static_assert(SC_THREADS == 256, "the transform's workgroups are 256 threads");
template <int NB, int G, int VEC>
__global__ __launch_bounds__(256) void k_transform_fixup(const float* __restrict__ X, int64_t M, int K,
                                                         const float4* __restrict__ Wp, int NBP, int Nc,
                                                         const float* __restrict__ rscale, float* __restrict__ Y,
                                                         int gx, int gblocks, int stream, ScatterParams p,
                                                         const int4* __restrict__ fix, int64_t nfix) {
    __shared__ PanelLds<TAURUS_F32, NB> lds;
    const int b = (int)blockIdx.x;
    if (b < gblocks) {
        gemm_panel_block<TAURUS_F32, NB>(X, M, K, Wp, NBP, Nc, rscale, Y, b % gx, b / gx, lds, stream != 0,
                                         SelfFlush{});
        return;
    }
    fixup_rows<G, VEC>(p, fix, nfix, b - gblocks);
}

static void transform_with_fixup(const ScatterShape& sh, const float* X, int64_t M, int K, const float* Wp, int Nc,
                                 const float* rscale, float* Y, const ScatterParams& p, const int4* fix,
                                 int64_t nfix, hipStream_t s) {
    const int NBP = gemm_packed_blocks_n(Nc);
    const int nb = NBP <= 4 ? 4 : 8;
    const int gx = (int)ceil_div(M, PANEL_ROWS), gy = (int)ceil_div(NBP, nb);
    const int64_t fblocks = ceil_div(nfix, SC_THREADS / sh.G);
    const int64_t blocks = (int64_t)gx * gy + fblocks;
    if (blocks >= ((int64_t)1 << 31)) fail(TAURUS_E_INVALID, "transform of %lld rows is too large", (long long)M);
    const float4* w = reinterpret_cast<const float4*>(Wp);
    const int stream = transform_streams(M, Nc) ? 1 : 0;
#define TAURUS_CASE(g, v)                                                                                  \
    if (sh.G == g && sh.VEC == v) {                                                                        \
        if (nb == 4)                                                                                       \
            k_transform_fixup<4, g, v><<<(unsigned)blocks, 256, 0, s>>>(X, M, K, w, NBP, Nc, rscale, Y, gx,  \
                                                                       gx * gy, stream, p, fix, nfix);     \
        else                                                                                               \
            k_transform_fixup<8, g, v><<<(unsigned)blocks, 256, 0, s>>>(X, M, K, w, NBP, Nc, rscale, Y, gx,  \
                                                                       gx * gy, stream, p, fix, nfix);     \
        TAURUS_CHECK_LAUNCH();                                                                             \
        return;                                                                                            \
    }
    TAURUS_ROW_SHAPES(TAURUS_CASE)
#undef TAURUS_CASE
    fail(TAURUS_E_INVALID, "unsupported row shape G=%d VEC=%d", sh.G, sh.VEC);
}

static void push_chunk(taurus_layer* L, int64_t b, int64_t e, const void* x, int32_t x_on_host) {
    if (L->poisoned) fail(TAURUS_E_STATE, "layer handle is poisoned by an earlier failure");
    if (b < 0 || e > L->n || b >= e || b % L->C != 0 || e != std::min(b + L->C, L->n))
        fail(TAURUS_E_INVALID, "chunk [%lld, %lld) is not a whole chunk of size %lld",
             (long long)b, (long long)e, (long long)L->C);
    if (!x) fail(TAURUS_E_INVALID, "x is null");
    if (x_on_host != 0 && x_on_host != 1) fail(TAURUS_E_INVALID, "x_on_host=%d", x_on_host);
    const int64_t k = b / L->C;
    if (L->pushed[(size_t)k]) fail(TAURUS_E_STATE, "chunk %lld pushed twice", (long long)k);
    if (L->acc_deferred) {
        L->acc = L->arena.alloc<float>(L->n * (int64_t)L->d_o, "accumulators");
        L->acc_deferred = false;
    }
    const ChunkIndex& idx = *L->idx;
    hipStream_t s = L->s;
    if (x_on_host) x = stage_host_chunk(L, x, e - b);
    // profile 1: events around every kernel; profile 2: around the scatter
    // launch only (ev[1] and ev[2])
    hipEvent_t ev[EV_PER_CHUNK] = {};
    if (L->d.profile) {
        for (int i = 0; i < EV_PER_CHUNK; i++)
            if (L->d.profile == 1 || i == 1 || i == 2) ev[i] = L->events[(size_t)k * EV_PER_CHUNK + i];
        if (ev[0]) TAURUS_HIP(hipEventRecord(ev[0], s));
    }
    L->pushed[(size_t)k] = 1;
    L->npushed++;
    ResChunk rc{};
    if (L->res) {
        for (int l = 0; l < RES_LISTS; l++) {
            rc.u[l] = idx.list_at(l, k);
            rc.n[l] = idx.list_count(l, k);
        }
        rc.first_row = b;
        rc.rows = e - b;
        L->res->prepare(rc, (int32_t)k, L->cnt, s);
    }
    const float* rscale = L->n_out ? L->n_out + b : nullptr;
    // GAT: the first pass only, into the layer's table of transformed rows
    float* ydst = L->gat_hp ? L->gat_hp + b * (int64_t)L->ncols : L->Y;
    SelfFlush sf{};
    if (L->self_in_transform) {
        sf.own = idx.has_own;
        sf.cnt = L->cnt;
        sf.acc = L->acc;
        sf.out = L->out_dev;
        sf.bias = L->bias;
        sf.first_row = b;
        sf.self_col = L->d_o;
        sf.d_o = L->d_o;
        sf.relu = L->d.relu;
        sf.out_dtype = L->d.out_dtype;
    }
    const SelfFlush* sfp = L->self_in_transform ? &sf : nullptr;
    if (L->d.in_dtype == TAURUS_F32 && L->fix_pending) {
        transform_with_fixup(L->shape, static_cast<const float*>(x), e - b, L->d.d_in, L->wpack, L->ystride, rscale,
                             ydst, L->fix_p, L->fix_list, L->fix_n, s);
        L->fix_pending = false;
    } else if (L->d.in_dtype == TAURUS_F32)
        gemm_f32(static_cast<const float*>(x), e - b, L->d.d_in, L->wpack, L->ystride, rscale, ydst, sfp, s);
    else
        gemm_16(static_cast<const uint16_t*>(x), L->d.in_dtype, e - b, L->d.d_in,
                static_cast<const uint16_t*>(L->wpack_any), L->ystride, rscale, ydst, sfp, s);
    if (x_on_host) TAURUS_HIP(hipEventRecord(L->gemm_done[(L->host_pushes - 1) & 1], s));
    if (ev[1]) TAURUS_HIP(hipEventRecord(ev[1], s));
    if (L->gat_hp) {  // the attention terms of the chunk's rows; passes 2 and 3 run at finalize
        k_gat_scores<<<(unsigned)ceil_div(e - b, 4), 256, 0, s>>>(ydst, e - b, L->ncols, L->d_o, L->gat_attn);
        TAURUS_CHECK_LAUNCH();
        if (ev[2]) TAURUS_HIP(hipEventRecord(ev[2], s));
        if (ev[3]) TAURUS_HIP(hipEventRecord(ev[3], s));
        return;
    }
    ScatterParams p{};
    p.Y = L->Y;
    p.ystride = L->ystride;
    p.self_col = L->d.agg == TAURUS_SAGE_MEAN ? L->d_o : 0;
    p.y_bytes = (int)(std::min(L->C, L->n) * (int64_t)L->ystride * 4);
    p.src = idx.item_src ? idx.item_src + idx.chunk_off[(size_t)k] : nullptr;
    p.has_own = idx.has_own;
    p.cnt = L->cnt;
    p.acc = L->res ? L->res->pool : L->acc;
    p.slot = L->res ? L->res->slot_of : nullptr;
    p.d_o = L->d_o;
    p.agg = L->d.agg;
    p.relu = L->d.relu;
    p.out_dtype = L->d.out_dtype;
    p.bias = L->bias;
    p.out = L->out_dev;
    p.carry = L->carry;
    p.carry_cnt = L->carry_cnt;
    p.long_base = idx.list_off[NCLASS][(size_t)k];
    p.first_row = b;
    p.rows = e - b;
    p.self_done = L->self_in_transform ? 1 : 0;
    p.self_tally = L->self_tally;
    ChunkUnits cu;
    for (int l = 0; l <= NCLASS; l++) {
        cu.u[l] = idx.list_at(l, k);
        cu.n[l] = idx.list_count(l, k);
    }
    dispatch_scatter(L->shape, p, cu, s);
    if (ev[2]) TAURUS_HIP(hipEventRecord(ev[2], s));
    const int64_t nfix = idx.list_count(NCLASS + 1, k);
    if (nfix > 0 && L->fuse_fix) {
        L->fix_p = p;
        L->fix_list = idx.list_at(NCLASS + 1, k);
        L->fix_n = nfix;
        L->fix_pending = true;
    } else if (nfix > 0) {
        dispatch_fixup(L->shape, p, idx.list_at(NCLASS + 1, k), nfix, s);
    }
    if (L->comp_ids) {
        // the destinations that completed in this chunk's scatter and fix-up
        const int64_t c0 = L->comp_off[(size_t)k], M = L->comp_off[(size_t)k + 1] - c0;
        const int nbp = gemm_packed_blocks_n(L->d.d_out);
        const int64_t tiles = ceil_div(M, PANEL_ROWS) * ceil_div(nbp, GRAD_NB);
        if (tiles > 0) {
            k_graduate<<<(unsigned)std::min<int64_t>(tiles, L->grad_blocks), 256, 0, s>>>(
                L->acc, L->d_o, reinterpret_cast<const float4*>(L->w2pack), nbp, L->d.d_out, L->comp_ids + c0, M,
                L->bias2, L->out_dev, L->d.out_dtype, L->d.relu);
            TAURUS_CHECK_LAUNCH();
        }
    }
    if (ev[3]) TAURUS_HIP(hipEventRecord(ev[3], s));
    if (L->res) L->res->release(rc, L->cnt, s);
}

// GAT passes 2 (softmax statistics) and 3 (aggregation) over every chunk,
// in chunk order, once all chunks are transformed
static void run_gat_passes(taurus_layer* L) {
    hipStream_t s = L->s;
    const ChunkIndex& idx = *L->idx;
    GatParams q;
    q.hp = L->gat_hp;
    q.ystride = L->ncols;
    q.d_o = L->d_o;
    q.m = L->gat_m;
    q.S = L->gat_s;
    q.scarry = L->gat_carry;
    auto params = [&](int64_t k) {
        const int64_t b = k * L->C, e = std::min(b + L->C, L->n);
        ScatterParams p{};
        p.Y = L->gat_hp + b * (int64_t)L->ncols;
        p.ystride = L->ncols;
        p.self_col = 0;
        p.y_bytes = (int)((e - b) * (int64_t)L->ncols * 4);
        p.src = idx.item_src ? idx.item_src + idx.chunk_off[(size_t)k] : nullptr;
        p.has_own = idx.has_own;
        p.cnt = L->cnt;
        p.acc = L->acc;
        p.slot = nullptr;
        p.d_o = L->d_o;
        p.agg = L->d.agg;
        p.relu = L->d.relu;
        p.out_dtype = L->d.out_dtype;
        p.bias = L->bias;
        p.out = L->out_dev;
        p.carry = L->carry;
        p.carry_cnt = L->carry_cnt;
        p.long_base = idx.list_off[NCLASS][(size_t)k];
        p.first_row = b;
        p.rows = e - b;
        p.att_t = L->gat_hp + L->d_o + 1;
        p.att_m = L->gat_m;
        p.att_s = L->gat_s;
        return p;
    };
    auto units = [&](int64_t k, int64_t& nshort) {
        ChunkUnits cu{};
        nshort = 0;
        for (int l = 0; l <= NCLASS; l++) {
            cu.u[l] = idx.list_at(l, k);
            cu.n[l] = idx.list_count(l, k);
            if (l < NCLASS) nshort += cu.n[l];
        }
        return cu;
    };
    const int T = 256;
    for (int64_t k = 0; k < L->nchunks; k++) {
        const ScatterParams p = params(k);
        int64_t nshort = 0;
        const ChunkUnits cu = units(k, nshort);
        if (nshort > 0) {
            k_gat_stats_short<<<(unsigned)ceil_div(nshort, T), T, 0, s>>>(p, cu, q, nshort);
            TAURUS_CHECK_LAUNCH();
        }
        if (cu.n[NCLASS] > 0) {
            k_gat_stats_pieces<<<(unsigned)ceil_div(cu.n[NCLASS], T / 64), T, 0, s>>>(p, cu.u[NCLASS], cu.n[NCLASS], q);
            TAURUS_CHECK_LAUNCH();
        }
        k_gat_stats_self<<<(unsigned)ceil_div(p.rows, T), T, 0, s>>>(p, q);
        TAURUS_CHECK_LAUNCH();
        const int64_t nfix = idx.list_count(NCLASS + 1, k);
        if (nfix > 0) {
            k_gat_stats_fixup<<<(unsigned)ceil_div(nfix, T), T, 0, s>>>(p, idx.list_at(NCLASS + 1, k), nfix, q);
            TAURUS_CHECK_LAUNCH();
        }
    }
    for (int64_t k = 0; k < L->nchunks; k++) {
        const ScatterParams p = params(k);
        int64_t nshort = 0;
        const ChunkUnits cu = units(k, nshort);
        dispatch_scatter(L->shape, p, cu, s, true);
        const int64_t nfix = idx.list_count(NCLASS + 1, k);
        if (nfix > 0) dispatch_fixup(L->shape, p, idx.list_at(NCLASS + 1, k), nfix, s);
    }
    L->gat_done = true;
}

static int finalize(taurus_layer* L, taurus_stats* st) {
    if (L->poisoned) fail(TAURUS_E_STATE, "layer handle is poisoned by an earlier failure");
    hipStream_t s = L->s;
    const ChunkIndex& idx = *L->idx;
    if (L->fix_pending) {  // the last chunk's fix-up
        dispatch_fixup(L->shape, L->fix_p, L->fix_list, L->fix_n, s);
        L->fix_pending = false;
    }
    if (L->gat_hp && !L->gat_done && L->npushed == L->nchunks) run_gat_passes(L);
    Arena tmp(s);
    unsigned long long* dleft = tmp.alloc<unsigned long long>(1, "pending count");
    fill_i32(reinterpret_cast<int32_t*>(dleft), 2, 0, s);
    k_count_pending<<<(unsigned)ceil_div(L->n, 256), 256, 0, s>>>(L->cnt, L->n, dleft);
    TAURUS_CHECK_LAUNCH();
    unsigned long long left = 0, own = 0;
    std::vector<unsigned long long> tally(L->self_tally ? 2 * TALLY_SLOTS : 0);
    Readback rb;
    rb.add(&left, dleft, 1);
    rb.add(&own, idx.own_count, 1);
    if (L->self_tally) rb.add(tally.data(), L->self_tally, 2 * TALLY_SLOTS);
    rb.run(s);
    if (st) {
        std::memset(st, 0, sizeof(*st));
        st->n = L->n;
        st->e = L->g.e;
        st->messages = idx.kept;
        st->self_terms = L->n;
        st->pairs = idx.segments + L->n - (int64_t)own;  // own-chunk segments carry their vertex's self message
        if (L->self_in_transform) {
            st->self_in_transform = L->n - (int64_t)own;
            st->self_fresh = st->self_last = L->self_tally ? 0 : -1;  // -1: not counted
        }
        for (int i = 0; i < (int)tally.size(); i += 2) {
            st->self_fresh += (int64_t)tally[(size_t)i];
            st->self_last += (int64_t)tally[(size_t)i + 1];
        }
        st->pending_left = (int64_t)left;
        st->completed = L->n - (int64_t)left;
        st->chunks = L->nchunks;
        st->chunks_pushed = L->npushed;
        for (int c = 0; c < NCLASS; c++) st->short_units += idx.n_list[c];
        st->wave_units = idx.n_list[NCLASS];
        st->split_segments = idx.n_list[NCLASS + 1];
        st->device_bytes = L->arena.peak() + (L->ms_index > 0 ? idx.arena.peak() : 0);
        st->ms_init = L->ms_init;
        st->ms_index = L->ms_index;
        const int64_t row_bytes = (int64_t)L->d_o * 4;
        const int64_t out_bytes = (int64_t)L->d_o * (L->d.out_dtype == TAURUS_F32 ? 4 : 2);
        if (L->res) {
            st->evictions = L->res->evictions;
            st->reloads = L->res->reload_count(s);
            st->hub_message_share = L->res->hub_share;
            st->device_bytes += L->res->arena.peak();
            st->pool_rows = L->res->S;
            st->hub_rows = L->res->H;
        }
        st->h2d_bytes = L->h2d_bytes + st->reloads * row_bytes;
        st->d2h_bytes = st->evictions * row_bytes + (L->d.out_on_host ? (L->n - (int64_t)left) * out_bytes : 0);
        for (int64_t k = 0; k < L->nchunks && !L->events.empty(); k++) {
            if (!L->pushed[(size_t)k]) continue;
            hipEvent_t* ev = &L->events[(size_t)k * EV_PER_CHUNK];
            float t[EV_PER_CHUNK - 1] = {};
            for (int i = 0; i + 1 < EV_PER_CHUNK; i++)
                if (L->d.profile == 1 || i == 1) TAURUS_HIP(hipEventElapsedTime(&t[i], ev[i], ev[i + 1]));
            st->ms_gemm += t[0];
            st->ms_scatter += t[1];
            st->ms_fixup += t[2];
            st->launches_gemm++;
            st->launches_scatter++;
            st->launches_fixup += idx.list_count(NCLASS + 1, k) > 0 ? 1 : 0;
        }
    }
    return left ? TAURUS_E_INCOMPLETE : TAURUS_OK;
}

int reorder_impl(const taurus_graph& g, int32_t* new_of_old, hipStream_t s);
int reorder_rcm_impl(const taurus_graph& g, int32_t* new_of_old, hipStream_t s);
int reorder_ta_impl(const taurus_graph& g, const int32_t* pi0, int iters, int32_t* pi, double* positions,
                    int64_t* spans, double* disp, int32_t* done, hipStream_t s);
int relabel_impl(const taurus_graph& g, const int32_t* new_of_old, int64_t* row_off, int32_t* col_dst,
                 hipStream_t s);
int permute_rows_impl(const void* in, void* out, int64_t n, int64_t row_bytes, const int32_t* new_of_old,
                      int inverse, hipStream_t s);

// ------------------------------------------------------------ loader -----
// Chunk j is filled into ring buffer j % R by whichever loader thread takes
// it (threads take chunks in ascending order), once the chunk R before it
// has left that buffer.  The calling thread pushes chunk j once it is
// filled; push_chunk(j) returns only after chunk j - 1's copy to the device
// is done (stage_host_chunk), which releases chunk j - 1's buffer.
struct HostRing {  // from the pinned block cache
    void* p = nullptr;
    size_t cap = 0;
    ~HostRing() { pinned_return(p, cap); }
};

static void stream_layer(taurus_layer* L, taurus_fill_fn fill, void* ctx, int threads, int ring,
                         taurus_stream_stats* st) {
    const auto t0 = std::chrono::steady_clock::now();
    if (L->poisoned) fail(TAURUS_E_STATE, "layer handle is poisoned by an earlier failure");
    if (!fill) fail(TAURUS_E_INVALID, "fill is null");
    if (threads < 1 || threads > 64) fail(TAURUS_E_INVALID, "threads=%d outside [1, 64]", threads);
    if (ring == 0) ring = 2 * threads;
    if (ring < threads + 1 || ring > 256) fail(TAURUS_E_INVALID, "ring=%d outside [threads + 1, 256]", ring);
    if (L->npushed != 0) fail(TAURUS_E_STATE, "the loader pushes every chunk; %lld were pushed before",
                              (long long)L->npushed);
    const int64_t nch = L->nchunks, C = L->C;
    const size_t row = (size_t)L->d.d_in * (L->d.in_dtype == TAURUS_F32 ? 4 : 2);
    const size_t slot = (size_t)std::min(C, L->n) * row;
    HostRing buf;
    buf.p = pinned_acquire(std::max<size_t>(1, slot) * (size_t)ring, &buf.cap);
    auto at = [&](int64_t j) { return static_cast<char*>(buf.p) + (size_t)(j % ring) * slot; };

    std::mutex m;
    std::condition_variable cv;
    int64_t next = 0;                         // next chunk a loader thread takes
    int64_t released = 0;                     // chunks [0, released) have left the ring
    std::vector<int64_t> ready((size_t)ring, -1);  // chunk filled into each buffer
    bool stop = false;
    int64_t bad_chunk = -1;
    int bad_rc = 0;
    std::atomic<int64_t> fill_ns{0};
    auto worker = [&]() {
        for (;;) {
            int64_t j;
            {
                std::unique_lock<std::mutex> lk(m);
                cv.wait(lk, [&] { return stop || next >= nch || released > next - ring; });
                if (stop || next >= nch) return;
                j = next++;
            }
            const int64_t b = j * C, e = std::min(b + C, L->n);
            const auto f0 = std::chrono::steady_clock::now();
            const int rc = fill(ctx, b, e, at(j));
            fill_ns += std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now() - f0)
                           .count();
            std::lock_guard<std::mutex> lk(m);
            if (rc != 0) {
                if (bad_chunk < 0) {
                    bad_chunk = j;
                    bad_rc = rc;
                }
                stop = true;
            } else {
                ready[(size_t)(j % ring)] = j;
            }
            cv.notify_all();
        }
    };
    std::vector<std::thread> pool;
    auto halt = [&]() {
        {
            std::lock_guard<std::mutex> lk(m);
            stop = true;
        }
        cv.notify_all();
        for (auto& t : pool) t.join();
        pool.clear();
    };
    double wait_s = 0, push_s = 0;
    try {
        for (int i = 0; i < threads; i++) pool.emplace_back(worker);
        for (int64_t j = 0; j < nch; j++) {
            const auto w0 = std::chrono::steady_clock::now();
            {
                std::unique_lock<std::mutex> lk(m);
                cv.wait(lk, [&] { return stop || ready[(size_t)(j % ring)] == j; });
                if (ready[(size_t)(j % ring)] != j) break;  // a fill failed
            }
            const auto p0 = std::chrono::steady_clock::now();
            wait_s += std::chrono::duration<double>(p0 - w0).count();
            push_chunk(L, j * C, std::min(j * C + C, L->n), at(j), 1);
            push_s += std::chrono::duration<double>(std::chrono::steady_clock::now() - p0).count();
            {  // chunk j - 1's copy is done: its buffer is free
                std::lock_guard<std::mutex> lk(m);
                if (j > 0) ready[(size_t)((j - 1) % ring)] = -1;
                released = j;
            }
            cv.notify_all();
        }
        // the last chunk's copy leaves the ring before the ring is freed
        for (int i = 0; i < 2; i++)
            if (L->stage_used[i]) TAURUS_HIP(hipEventSynchronize(L->h2d_done[i]));
    } catch (...) {
        halt();
        // copies from the ring may still be queued: let them finish before
        // the ring is freed
        if (L->copy_stream) (void)hipStreamSynchronize(L->copy_stream);
        throw;
    }
    halt();
    if (bad_chunk >= 0) {
        L->poisoned = true;
        fail(TAURUS_E_INVALID, "fill returned %d for chunk %lld", bad_rc, (long long)bad_chunk);
    }
    if (st) {
        st->chunks = nch;
        st->bytes = (int64_t)row * L->n;
        st->fill_seconds = (double)fill_ns.load() * 1e-9;
        st->wait_seconds = wait_s;
        st->push_seconds = push_s;
        st->wall_seconds = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    }
}

// Runs an entry point's body: library failures become their status, any
// other exception TAURUS_E_DEVICE; nothing crosses the C boundary.
template <typename F>
static int guarded(F&& f) {
    try {
        return f();
    } catch (const Failure& x) {
        return x.status;
    } catch (const std::exception& x) {
        set_error("internal error: %s", x.what());
        return TAURUS_E_DEVICE;
    }
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

int taurus_build_csr_noalloc(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                             int32_t* col_dst, void* stream) {
    try {
        return build_csr_noalloc_impl(n, e, src, dst, row_off, col_dst, static_cast<hipStream_t>(stream));
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
        (void)stream;  // structures are built by the first layer that uses them, on its stream
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

int taurus_reorder(const taurus_graph* g, int32_t* new_of_old, void* stream) {
    return guarded([&] {
        check_graph_args(g);
        if (!new_of_old) fail(TAURUS_E_INVALID, "new_of_old is null");
        return reorder_impl(*g, new_of_old, static_cast<hipStream_t>(stream));
    });
}

int taurus_reorder_rcm(const taurus_graph* g, int32_t* new_of_old, void* stream) {
    return guarded([&] {
        check_graph_args(g);
        if (!new_of_old) fail(TAURUS_E_INVALID, "new_of_old is null");
        return reorder_rcm_impl(*g, new_of_old, static_cast<hipStream_t>(stream));
    });
}

int taurus_reorder_ta(const taurus_graph* g, const int32_t* pi0, int32_t iterations, int32_t* new_of_old,
                      double* positions, int64_t* spans, double* disp, int32_t* updates, void* stream) {
    return guarded([&] {
        check_graph_args(g);
        if (!new_of_old) fail(TAURUS_E_INVALID, "new_of_old is null");
        if (iterations < 1) fail(TAURUS_E_INVALID, "iterations=%d, at least 1", (int)iterations);
        int32_t done = 0;
        const int rc = reorder_ta_impl(*g, pi0, iterations, new_of_old, positions, spans, disp, &done,
                                       static_cast<hipStream_t>(stream));
        if (updates) *updates = done;
        return rc;
    });
}

int taurus_relabel_graph(const taurus_graph* g, const int32_t* new_of_old, int64_t* row_off, int32_t* col_dst,
                         void* stream) {
    return guarded([&] {
        check_graph_args(g);
        if (!new_of_old || !row_off || (g->e > 0 && !col_dst)) fail(TAURUS_E_INVALID, "null output or permutation");
        return relabel_impl(*g, new_of_old, row_off, col_dst, static_cast<hipStream_t>(stream));
    });
}

int taurus_permute_rows(const void* in, void* out, int64_t n, int64_t row_bytes, const int32_t* new_of_old,
                        int32_t inverse, void* stream) {
    return guarded([&] {
        if (n <= 0 || n >= ((int64_t)1 << 31)) fail(TAURUS_E_INVALID, "n=%lld out of range", (long long)n);
        if (row_bytes <= 0 || row_bytes % 4) fail(TAURUS_E_INVALID, "row_bytes=%lld: a positive multiple of 4",
                                                  (long long)row_bytes);
        if (!in || !out || !new_of_old) fail(TAURUS_E_INVALID, "null pointer");
        if (in == out) fail(TAURUS_E_INVALID, "in and out must not overlap");
        if (inverse != 0 && inverse != 1) fail(TAURUS_E_INVALID, "inverse=%d", inverse);
        return permute_rows_impl(in, out, n, row_bytes, new_of_old, inverse, static_cast<hipStream_t>(stream));
    });
}

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
        // argument errors leave the handle as it was; a failure once the
        // chunk's work has started poisons it
        if (f.status == TAURUS_E_OOM || f.status == TAURUS_E_DEVICE || f.status == TAURUS_E_BUDGET)
            L->poisoned = true;
        return f.status;
    }
}

int taurus_stream_layer(taurus_layer* L, taurus_fill_fn fill, void* ctx, int32_t threads, int32_t ring,
                        taurus_stream_stats* stats) {
    if (!L) {
        set_error("null layer handle");
        return TAURUS_E_INVALID;
    }
    try {
        stream_layer(L, fill, ctx, threads, ring, stats);
        return TAURUS_OK;
    } catch (const Failure& f) {
        if (f.status == TAURUS_E_OOM || f.status == TAURUS_E_DEVICE || f.status == TAURUS_E_BUDGET)
            L->poisoned = true;
        return f.status;
    } catch (const std::exception& x) {
        L->poisoned = true;
        set_error("internal error: %s", x.what());
        return TAURUS_E_DEVICE;
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
        if (L->csc && !L->mask && words > 0) {
            L->mask = L->arena.alloc<uint64_t>(words, "fanout mask");
            sample_mask(L->g, *L->csc, L->d.seed, L->d.layer, L->d.fanout, L->mask, L->s);
        }
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

int64_t taurus_release_cached_memory(int64_t bytes) {
    try {
        release_pinned();
        return (int64_t)release_cached(bytes <= 0 ? 0 : (size_t)bytes);
    } catch (const Failure& f) {
        return f.status;
    }
}

int taurus_layer_reload_histogram(taurus_layer* L, int64_t* counts, int32_t bins) {
    if (!L || !counts || bins < 2) {
        set_error("null argument or bins < 2");
        return TAURUS_E_INVALID;
    }
    try {
        if (L->res) {
            L->res->reload_histogram(counts, bins, L->s);
        } else {
            for (int b = 0; b < bins; b++) counts[b] = 0;
            counts[0] = L->n;
        }
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
