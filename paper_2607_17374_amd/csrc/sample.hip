// Fanout sampling (Sec. 3.9, "Sampling-based Inference"): for every
// destination v keep the min(d_in(v), k) in-edges (u, v) whose rank pairs
// (H(seed, 4, layer, v, u), u) are smallest; the rest do not propagate in
// this layer.
//
// The in-edges of each destination are read from a CSC, built once per
// graph by a stable radix sort of the CSR edges by destination (sources stay
// ascending within a destination).  Per layer one pass over the in-lists
// decides every in-edge and writes the kept ones straight out, in CSC order,
// at position koff[v] + (kept in-edges of v before it), koff = the exclusive
// scan of min(d_in, k):
//   - lists of at most min(k, 64) in-edges are kept whole: a wave copies the
//     lists of 64 consecutive destinations in-edge-parallel;
//   - lists of k+1 .. 64 in-edges (collected by that pass): 16 lanes per
//     destination hold the whole list (4 in-edges a lane); an in-edge is
//     kept iff fewer than k pairs of its list are smaller (every pair is
//     compared with every other by broadcast within the 16 lanes);
//   - longer lists: a wave each.  Keys are uniform 64-bit values, so the k
//     smallest lie below a cutoff that passes about k + 4 sqrt(k) + 16 of
//     them; the wave counts the keys at or below a cutoff, moves it until
//     between k and a cap (256 or 1024) pass (SplitMix64's finaliser is a
//     bijection, so one destination's keys are distinct and the count rises
//     by one key at a time: some cutoff always qualifies), gathers those
//     candidates in LDS and ranks them by pairwise comparison.  Every pair
//     below the k-th smallest passes any qualifying cutoff, so the kept set
//     is exact.
// Rank pairs are distinct within a destination (the sources are), so the
// kept set is unique.  The same pass can instead set the kept edges' bits
// in a CSR-order mask (each kept (u, v) found in row u by binary search),
// for callers that want the mask.
#include "device.hpp"
#include "internal.hpp"

namespace taurus {

// ------------------------------------------------------------------ CSC ----
__global__ void k_validate_csr(const int64_t* __restrict__ row_off, const int32_t* __restrict__ col_dst,
                               int64_t n, int64_t e, int* __restrict__ bad) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i == 0 && (row_off[0] != 0 || row_off[n] != e)) atomicOr(bad, 1);
    if (i < n && row_off[i] > row_off[i + 1]) atomicOr(bad, 1);
    if (i < e) {
        const int32_t c = col_dst[i];
        if (c < 0 || (int64_t)c >= n) atomicOr(bad, 2);
    }
}

void validate_csr(const taurus_graph& g, hipStream_t s) {
    Arena tmp(s);
    int* bad = tmp.alloc<int>(1, "graph flag");
    fill_i32(bad, 1, 0, s);
    k_validate_csr<<<(unsigned)ceil_div(std::max(std::max(g.n, g.e), (int64_t)1), 256), 256, 0, s>>>(
        g.row_off, g.col_dst, g.n, g.e, bad);
    TAURUS_CHECK_LAUNCH();
    int hbad = 0;
    Readback rb;
    rb.add(&hbad, bad, 1);
    rb.run(s);
    if (hbad) fail(TAURUS_E_INVALID, "graph is not a valid CSR over [0, n) (flags %d)", hbad);
}

// CSR edge i -> sort key v, value u; flags a row that is not strictly
// ascending or holds a self loop (bit 16).  A workgroup takes CI_TILE
// consecutive edges and finds their rows through tile_rows.
constexpr int CI_ITEMS = 16, CI_TILE = 256 * CI_ITEMS, CI_ROWS = 8192;
__global__ __launch_bounds__(256) void k_csc_items(const int64_t* __restrict__ row_off,
                                                   const int32_t* __restrict__ col_dst, int64_t n, int64_t e,
                                                   uint32_t* __restrict__ keys, uint32_t* __restrict__ vals,
                                                   int* __restrict__ bad) {
    __shared__ int32_t ro[CI_ROWS + 1];
    __shared__ int64_t bnd[2];
    const int64_t i0 = (int64_t)blockIdx.x * CI_TILE, i1 = min(i0 + CI_TILE, e);
    const TileRows t = tile_rows<CI_ROWS, CI_TILE>(row_off, n, i0, i1, ro, bnd);
    bool flag = false;
#pragma unroll 4
    for (int r = 0; r < CI_ITEMS; r++) {
        const int64_t i = i0 + (int64_t)r * 256 + threadIdx.x;
        if (i >= i1) break;
        bool later;
        const int64_t u = tile_row_of(t, row_off, ro, i0, i, later);
        const int32_t v = col_dst[i];
        if ((int64_t)v == u || (later && col_dst[i - 1] >= v)) flag = true;
        keys[i] = (uint32_t)v;
        vals[i] = (uint32_t)u;
    }
    if (flag) atomicOr(bad, 16);
}

// destinations with more than 64 in-edges (the long-list sampling pass)
__global__ void k_heavy_flags(const int64_t* __restrict__ in_off, int64_t n, int32_t* __restrict__ flag) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n) flag[v] = in_off[v + 1] - in_off[v] > 64 ? 1 : 0;
}
__global__ void k_heavy_list(const int32_t* __restrict__ flag, const int64_t* __restrict__ pos, int64_t n,
                             int32_t* __restrict__ heavy) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n && flag[v]) heavy[pos[v]] = (int32_t)v;
}

// in_off from the sorted destinations (e >= 1; in_off filled with -1
// beforehand), as the CSR build's row offsets: position i starts its
// destination v when its predecessor's destination differs, and so every
// empty destination in between when there are at most CSC_GAP_INLINE; the
// last position ends the rest the same way.  Longer runs stay -1 for
// k_csc_offsets_fill.  Destinations are below n (the CSR was checked),
// clamped so that every write stays in [0, n].
constexpr int64_t CSC_GAP_INLINE = 16;
__global__ void k_csc_offsets(const uint32_t* __restrict__ keys, int64_t e, int64_t n, int64_t* __restrict__ in_off) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= e) return;
    const int64_t v = min((int64_t)keys[i], n - 1);
    const int64_t vp = i > 0 ? min((int64_t)keys[i - 1], n - 1) : -1;
    if (vp < v) {
        in_off[v] = i;
        if (v - vp <= CSC_GAP_INLINE)
            for (int64_t w = vp + 1; w < v; w++) in_off[w] = i;
    }
    if (i == e - 1) {
        in_off[n] = e;
        if (n - v <= CSC_GAP_INLINE)
            for (int64_t w = v + 1; w < n; w++) in_off[w] = e;
    }
}
// the destinations k_csc_offsets left at -1: first position >= v (binary search)
__global__ void k_csc_offsets_fill(const uint32_t* __restrict__ keys, int64_t e, int64_t n,
                                   int64_t* __restrict__ in_off) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v > n || in_off[v] >= 0) return;
    int64_t lo = 0, hi = e;
    while (lo < hi) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if ((int64_t)keys[mid] < v) lo = mid + 1;
        else hi = mid;
    }
    in_off[v] = lo;
}

std::shared_ptr<Csc> build_csc(const taurus_graph& g, hipStream_t s, Arena* scratch) {
    const auto t0 = std::chrono::steady_clock::now();
    auto c = std::make_shared<Csc>(s);
    const int64_t n = g.n, e = g.e;
    const int T = 256;
    validate_csr(g, s);
    Arena own(s);
    Arena& tmp = scratch ? *scratch : own;
    int* bad = tmp.alloc<int>(1, "sort flag");
    fill_i32(bad, 1, 0, s);
    int hbad = 0;
    c->in_off = c->arena.alloc<int64_t>(n + 1, "in-edge offsets");
    if (e > 0) {
        SortBuffers32 sb{{tmp.alloc<uint32_t>(e, "csc keys"), tmp.alloc<uint32_t>(e, "csc keys (ping-pong)")},
                       {c->arena.alloc<uint32_t>(e, "in-edge sources"),
                        c->arena.alloc<uint32_t>(e, "in-edge sources (ping-pong)")},
                       0};
        k_csc_items<<<(unsigned)ceil_div(e, CI_TILE), 256, 0, s>>>(g.row_off, g.col_dst, n, e, sb.keys[0],
                                                                  sb.vals[0], bad);
        TAURUS_CHECK_LAUNCH();
        radix_sort_u32(sb, e, std::max(1, bits_for(n - 1)), tmp, s, bad, 8);
        c->in_src = reinterpret_cast<int32_t*>(sb.vals[sb.cur]);
        c->arena.free_ptr(sb.vals[1 - sb.cur]);
        fill_i32(reinterpret_cast<int32_t*>(c->in_off), 2 * (n + 1), -1, s);
        k_csc_offsets<<<(unsigned)ceil_div(e, T), T, 0, s>>>(sb.keys[sb.cur], e, n, c->in_off);
        TAURUS_CHECK_LAUNCH();
        k_csc_offsets_fill<<<(unsigned)ceil_div(n + 1, T), T, 0, s>>>(sb.keys[sb.cur], e, n, c->in_off);
        TAURUS_CHECK_LAUNCH();
    } else {
        fill_i32(reinterpret_cast<int32_t*>(c->in_off), 2 * (n + 1), 0, s);
    }
    int32_t* flag = tmp.alloc<int32_t>(n, "long in-list flags");
    int64_t* pos = tmp.alloc<int64_t>(n + 1, "long in-list positions");
    k_heavy_flags<<<(unsigned)ceil_div(n, T), T, 0, s>>>(c->in_off, n, flag);
    TAURUS_CHECK_LAUNCH();
    scan_i32_to_i64(flag, pos, n, true, tmp, s);
    {
        Readback rb;
        rb.add(&hbad, bad, 1);
        rb.add(&c->nheavy, pos + n, 1);
        rb.run(s);
    }
    if (hbad & 16) fail(TAURUS_E_INVALID, "graph rows are not strictly ascending or hold a self loop");
    if (hbad) fail(TAURUS_E_DEVICE, "in-edge sort: radix offset out of range");
    if (c->nheavy > 0) {
        c->heavy = c->arena.alloc<int32_t>(c->nheavy, "long in-lists");
        k_heavy_list<<<(unsigned)ceil_div(n, T), T, 0, s>>>(flag, pos, n, c->heavy);
        TAURUS_CHECK_LAUNCH();
    }
    c->ms_build = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    return c;
}

// --------------------------------------------------------------- sampling ----
__device__ inline bool pair_less(uint64_t ka, uint32_t ua, uint64_t kb, uint32_t ub) {
    return ka < kb || (ka == kb && ua < ub);
}

constexpr int LIGHT_MAX = 64;     // lists up to this long are ranked in registers
// candidates a wave of the long-list pass holds in LDS: 256 while the
// cutoff's target k + 4 sqrt(k) + 16 stays well inside it (k <= 128), else
// 1024 (fewer workgroups fit a CU)
constexpr int HEAVY_CAP = 1024;
constexpr int HEAVY_CAP_SMALL = 256, HEAVY_SMALL_K = 128;
constexpr int REG_MAX = 512;      // long lists up to this length are held in registers

// Where the kept in-edges go: chunk-index items at koff[v] + (position among
// v's kept in-edges) -- key (chunk(u) << vbits | v), value u - chunk(u)*C --
// or, when mask is set, bit (CSR position of (u, v)) of a CSR-order mask.
struct SampleOut {
    uint64_t* keys;
    uint32_t* vals;
    const int64_t* koff;
    int64_t C;
    int vbits;
    unsigned long long* mask;
    const int64_t* row_off;
    const int32_t* col_dst;
    int* bad;  // bit SAMPLE_BAD: a list the cutoff search could not settle (repeated sources)
    int32_t* first_chunk;  // items mode: chunk of v's first kept source (its smallest), or null
};
constexpr int SAMPLE_BAD = 32;

// Kept in-edge (u, v) at item position `at` (items mode: koff[v] + its
// position among v's kept in-edges; `first` when that position is 0).
// fcu: chunk of v's smallest kept source.
__device__ inline void emit_item(const SampleOut& o, int64_t v, uint32_t u, int64_t at, bool first, uint32_t fcu) {
    if (o.mask) {
        int64_t lo = o.row_off[u], hi = o.row_off[u + 1];  // (u, v) is an edge: v is in row u
        while (lo < hi) {
            const int64_t mid = lo + ((hi - lo) >> 1);
            if ((int64_t)o.col_dst[mid] < v) lo = mid + 1;
            else hi = mid;
        }
        atomicOr(&o.mask[lo >> 6], 1ull << (lo & 63));
    } else {
        const uint32_t cu = u / (uint32_t)o.C;  // u < 2^31 and C < 2^31
        // not the destination's first flush: a chunk after the earlier of
        // its first kept source's chunk and its own chunk
        const uint64_t nf = cu != min(fcu, (uint32_t)v / (uint32_t)o.C) ? 1 : 0;
        o.keys[at] = ((uint64_t)cu << (o.vbits + 1)) | (nf << o.vbits) | (uint64_t)v;
        o.vals[at] = u - cu * (uint32_t)o.C;
        if (first && o.first_chunk) o.first_chunk[v] = (int32_t)cu;
    }
}

__device__ inline void emit_kept(const SampleOut& o, int64_t v, uint32_t u, int64_t pos, uint32_t fcu) {
    emit_item(o, v, u, o.mask ? 0 : o.koff[v] + pos, pos == 0, fcu);
}

// Lists of 1 .. min(k, LIGHT_MAX) in-edges, kept whole, and the
// destinations whose lists need ranking (k < d_in <= LIGHT_MAX) noted in
// rank_list.  A wave takes 64 consecutive destinations, a lane each; their
// kept in-edges are copied in-edge-parallel (item t of the wave's run goes
// to the lane whose running count first exceeds t), so the in-lists are
// read and the items written contiguously.
__global__ __launch_bounds__(256) void k_sample_short(const int64_t* __restrict__ in_off,
                                                      const int32_t* __restrict__ in_src, int64_t n, int k,
                                                      SampleOut o, int32_t* __restrict__ rank_list,
                                                      unsigned int* __restrict__ rank_count) {
    // destinations to rank wait in a per-wave LDS buffer and leave it 64 at
    // a time, so the shared list count takes one atomic per 64 of them
    __shared__ int32_t rbuf[4][128];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t lt = (1ull << lane) - 1ull;
    const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
    const int64_t cmax = min((int64_t)k, (int64_t)LIGHT_MAX);
    auto flush = [&](int cnt) {  // the first cnt buffered entries to the list
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        unsigned int at = 0;
        if (lane == 0) at = atomicAdd(rank_count, (unsigned int)cnt);
        at = __shfl(at, 0);
        if (lane < cnt) rank_list[at + lane] = rbuf[w][lane];
    };
    int rn = 0;  // buffered entries (uniform over the wave)
    for (int64_t v0 = wave * 64; v0 < n; v0 += nwaves * 64) {  // uniform over the wave
        const int64_t v = v0 + lane;
        int64_t a = 0, d = 0;
        if (v < n) {
            a = in_off[v];
            d = in_off[v + 1] - a;
        }
        const bool rank = d > k && d <= LIGHT_MAX;
        const uint64_t rb = __ballot(rank);
        if (rb) {
            if (rank) rbuf[w][rn + __popcll(rb & lt)] = (int32_t)v;
            rn += __popcll(rb);
            if (rn >= 64) {
                flush(64);
                const int32_t rest = lane + 64 < rn ? rbuf[w][lane + 64] : 0;
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
                if (lane + 64 < rn) rbuf[w][lane] = rest;
                rn -= 64;
            }
        }
        const int cnt = d > 0 && d <= cmax ? (int)d : 0;
        int incl = cnt;
#pragma unroll
        for (int m = 1; m < 64; m <<= 1) {
            const int y = __shfl_up(incl, m, 64);
            if (lane >= m) incl += y;
        }
        const int total = __shfl(incl, 63);
        // a kept list's first in-edge is its smallest source
        const uint32_t fcu = cnt ? (uint32_t)in_src[a] / (uint32_t)o.C : 0u;
        const int64_t ko = cnt && !o.mask ? o.koff[v] : 0;
        for (int t0 = 0; t0 < total; t0 += 64) {  // uniform over the wave
            const int t = t0 + lane;
            // owner: the first lane whose running count exceeds t
            int lo = 0, hi = 63;
#pragma unroll
            for (int q = 0; q < 6; q++) {
                const int mid = (lo + hi) >> 1;
                const int x = __shfl(incl, mid);
                if (x > t) hi = mid;
                else lo = mid + 1;
            }
            const int pos = t - (__shfl(incl, lo) - __shfl(cnt, lo));
            const int64_t al = __shfl(a, lo), kl = __shfl(ko, lo);
            const uint32_t fl = __shfl(fcu, lo);
            if (t < total) emit_item(o, v0 + lo, (uint32_t)in_src[al + pos], kl + pos, pos == 0, fl);
        }
    }
    if (rn > 0) flush(rn);
}

// Lists of k < d_in <= LIGHT_MAX in-edges (rank_list[0 .. *rank_count)),
// 16 lanes per destination, four destinations per wave, waves striding
// over the list.  Lane j of a group holds slots j, j + 16, j + 32, j + 48
// of its destination's list.
__global__ __launch_bounds__(256) void k_sample_light(const int64_t* __restrict__ in_off,
                                                      const int32_t* __restrict__ in_src,
                                                      const int32_t* __restrict__ rank_list,
                                                      const unsigned int* __restrict__ rank_count, uint64_t seed,
                                                      int layer, int k, SampleOut o) {
    const int lane = threadIdx.x & 63, sub = lane & 15, grp = lane >> 4;
    const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
    const int64_t nr = *rank_count;
    for (int64_t base = wave * 4; base < nr; base += nwaves * 4) {  // uniform over the wave
        const int64_t v = base + grp < nr ? (int64_t)rank_list[base + grp] : -1;
        int64_t a = 0, d = 0;
        if (v >= 0) {
            a = in_off[v];
            d = in_off[v + 1] - a;
        }
        const bool mine = v >= 0 && d > 0 && d <= LIGHT_MAX;
        const bool rank = mine && d > k;
        const uint64_t pre = rank ? sample_prefix(seed, (uint64_t)layer, (uint64_t)v) : 0;
        uint32_t u[4];
        uint64_t key[4];
        bool valid[4];
#pragma unroll
        for (int t = 0; t < 4; t++) {
            const int sl = t * 16 + sub;
            valid[t] = mine && sl < d;
            u[t] = valid[t] ? (uint32_t)in_src[a + sl] : ~0u;
            key[t] = valid[t] && rank ? sample_key(pre, u[t]) : ~0ull;
        }
        int below[4] = {0, 0, 0, 0};
        // registers holding slots of a list to rank, over the wave
        const int tn = (__ballot(rank) != 0) + (__ballot(rank && d > 16) != 0) + (__ballot(rank && d > 32) != 0) +
                       (__ballot(rank && d > 48) != 0);
        // every group broadcasts its slots in turn; invalid slots hold
        // (~0, ~0), which is never below a valid pair
#pragma unroll
        for (int t = 0; t < 4; t++) {
            if (t >= tn) break;  // uniform over the wave
            for (int j = 0; j < 16; j++) {
                const uint32_t klo = __shfl((uint32_t)key[t], j, 16), khi = __shfl((uint32_t)(key[t] >> 32), j, 16);
                const uint32_t uj = __shfl(u[t], j, 16);
                const uint64_t kj = ((uint64_t)khi << 32) | klo;
#pragma unroll
                for (int q = 0; q < 4; q++)
                    if (q < tn) below[q] += pair_less(kj, uj, key[q], u[q]) ? 1 : 0;
            }
        }
        // kept slots in slot order (slot = t * 16 + sub): the position among
        // the destination's kept in-edges counts the kept slots before it
        int before = 0;
        const int64_t mk = min(d, (int64_t)k);  // kept in-edges of v (distinct pairs)
        // the smallest kept source (slot order is source order)
        uint32_t umin = ~0u;
#pragma unroll
        for (int t = 0; t < 4; t++)
            if (valid[t] && (!rank || below[t] < k)) umin = min(umin, u[t]);
#pragma unroll
        for (int x = 8; x >= 1; x >>= 1) umin = min(umin, (uint32_t)__shfl_xor(umin, x, 16));
        const uint32_t fcu = umin / (uint32_t)o.C;
#pragma unroll
        for (int t = 0; t < 4; t++) {
            const bool kept = valid[t] && (!rank || below[t] < k);
            const uint64_t bal = __ballot(kept);
            const uint32_t g16 = (uint32_t)(bal >> (grp * 16)) & 0xffffu;
            const int pos = before + __popc(g16 & ((1u << sub) - 1u));
            if (kept && pos < mk) emit_kept(o, v, u[t], pos, fcu);
            before += __popc(g16);
        }
    }
}

// Lists longer than LIGHT_MAX (heavy[0 .. nheavy)), a wave each; the four
// waves of a workgroup keep their candidates in separate LDS slices.
template <int CAP>
__global__ __launch_bounds__(256) void k_sample_heavy(const int64_t* __restrict__ in_off,
                                                      const int32_t* __restrict__ in_src,
                                                      const int32_t* __restrict__ heavy, int64_t nheavy,
                                                      uint64_t seed, int layer, int k, SampleOut o) {
    __shared__ uint64_t ckey[4][CAP];
    __shared__ uint32_t cu[4][CAP];
    __shared__ uint64_t kbits[4][CAP / 64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t lt = (1ull << lane) - 1ull;
    const int64_t wave = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
    for (int64_t h = wave; h < nheavy; h += nwaves) {  // uniform over the wave
        const int64_t v = heavy[h];
        const int64_t a = in_off[v], d = in_off[v + 1] - a;
        if (d <= k) {  // every in-edge is kept; the first is the smallest
            const uint32_t fcu = (uint32_t)in_src[a] / (uint32_t)o.C;
            for (int64_t sl = lane; sl < d; sl += 64) emit_kept(o, v, (uint32_t)in_src[a + sl], sl, fcu);
            continue;
        }
        const uint64_t pre = sample_prefix(seed, (uint64_t)layer, (uint64_t)v);
        // lists of up to REG_MAX in-edges are read once into registers
        const bool in_regs = d <= REG_MAX;
        uint64_t rk[REG_MAX / 64];
        uint32_t ru[REG_MAX / 64];
        if (in_regs) {
#pragma unroll
            for (int t = 0; t < REG_MAX / 64; t++) {
                const int64_t sl = t * 64 + lane;
                ru[t] = sl < d ? (uint32_t)in_src[a + sl] : ~0u;
            }
#pragma unroll
            for (int t = 0; t < REG_MAX / 64; t++) rk[t] = (int64_t)t * 64 + lane < d ? sample_key(pre, ru[t]) : ~0ull;
        }
        // Count the keys at or below cut; with gather, also write those
        // candidates to LDS in CSC order (sources ascending) while they fit.
        // Longer lists stream through in blocks of REG_MAX, all of a
        // block's loads in flight before its keys are hashed.
        auto scan = [&](uint64_t cut, bool gather) {
            int64_t c = 0;
            auto take = [&](bool in, uint64_t kk, uint32_t uu) {
                const uint64_t bal = __ballot(in);
                if (gather && in) {
                    const int64_t at = c + __popcll(bal & lt);
                    if (at < CAP) {
                        ckey[w][at] = kk;
                        cu[w][at] = uu;
                    }
                }
                c += __popcll(bal);
            };
            if (in_regs) {
#pragma unroll
                for (int t = 0; t < REG_MAX / 64; t++) take((int64_t)t * 64 + lane < d && rk[t] <= cut, rk[t], ru[t]);
                return c;
            }
            for (int64_t b0 = 0; b0 < d; b0 += REG_MAX) {  // uniform over the wave
                uint32_t uu[REG_MAX / 64];
#pragma unroll
                for (int t = 0; t < REG_MAX / 64; t++) {
                    const int64_t sl = b0 + t * 64 + lane;
                    uu[t] = sl < d ? (uint32_t)in_src[a + sl] : 0u;
                }
#pragma unroll
                for (int t = 0; t < REG_MAX / 64; t++) {
                    const bool ok = b0 + t * 64 + lane < d;
                    const uint64_t kk = ok ? sample_key(pre, uu[t]) : ~0ull;
                    take(ok && kk <= cut, kk, uu[t]);
                }
            }
            return c;
        };
        // cutoff: about k + 4 sqrt(k) + 16 keys of d pass, gathering on the
        // way; if the count falls outside [k, CAP], widen or narrow the
        // cutoff by counting alone, then gather once more
        const double want = (double)k + 4.0 * sqrt((double)k) + 16.0;
        uint64_t cut = want >= (double)d ? ~0ull : (uint64_t)(want / (double)d * 18446744073709551616.0);
        bool have_lo = false, have_hi = false;
        uint64_t lo = 0, hi = 0;  // count(lo) < k, count(hi) > CAP
        int64_t cnt = scan(cut, true);
        bool gathered = true;
        int rounds = 0;
        while ((cnt < k || cnt > CAP) && ++rounds <= 200) {
            if (cnt < k) {
                lo = cut;
                have_lo = true;
            } else {
                hi = cut;
                have_hi = true;
            }
            if (!have_hi) cut = cut > (~0ull >> 1) ? ~0ull : 2 * cut + 1;
            else if (!have_lo) cut = cut >> 1;
            else cut = lo + ((hi - lo) >> 1);
            cnt = scan(cut, false);
            gathered = false;
        }
        if (cnt < k || cnt > CAP) {  // only repeated sources make the count jump past the window
            if (lane == 0) atomicOr(o.bad, SAMPLE_BAD);
            continue;
        }
        if (!gathered) scan(cut, true);
        const int64_t m = cnt;
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        // rank each candidate among all; keep the k smallest, in candidate
        // order.  The kept flags go to LDS first: the first kept candidate
        // (the smallest kept source) decides every kept item's key.
        uint32_t fcu = ~0u;
        for (int64_t i0 = 0; i0 < m; i0 += 64) {
            const int64_t i = i0 + lane;
            bool kept = false;
            if (i < m) {
                const uint64_t ki = ckey[w][i];
                const uint32_t ui = cu[w][i];
                int r = 0;
                for (int64_t j = 0; j < m && r < k; j++) r += pair_less(ckey[w][j], cu[w][j], ki, ui) ? 1 : 0;
                kept = r < k;
            }
            const uint64_t bal = __ballot(kept);
            if (lane == 0) kbits[w][i0 >> 6] = bal;
            if (bal && fcu == ~0u) fcu = cu[w][i0 + __builtin_ctzll(bal)] / (uint32_t)o.C;
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        int64_t before = 0;
        for (int64_t i0 = 0; i0 < m; i0 += 64) {
            const int64_t i = i0 + lane;
            const uint64_t bal = kbits[w][i0 >> 6];
            const bool kept = (bal >> lane) & 1;
            const int64_t pos = before + __popcll(bal & lt);
            if (kept && pos < k) emit_kept(o, v, cu[w][i], pos, fcu);
            before += __popcll(bal);
        }
        // the slice is rewritten by this wave's next destination
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    }
}

static void sample_pass(const Csc& csc, int64_t n, uint64_t seed, int layer, int k, const SampleOut& o,
                        Arena& tmp, hipStream_t s) {
    if (k < 1 || k > FANOUT_MAX) fail(TAURUS_E_INVALID, "fanout %d outside [1, %d]", k, FANOUT_MAX);
    if (n >= ((int64_t)1 << 31)) fail(TAURUS_E_INVALID, "sampler: %lld vertices exceed 2^31", (long long)n);
    int dev = 0, cus = 0;
    TAURUS_HIP(hipGetDevice(&dev));
    TAURUS_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    int32_t* rank_list = tmp.alloc<int32_t>(std::max<int64_t>(1, n), "short lists to rank");
    unsigned int* rank_count = tmp.alloc<unsigned int>(1, "short lists to rank: count");
    fill_i32(reinterpret_cast<int32_t*>(rank_count), 1, 0, s);
    const int64_t grid_short = std::min<int64_t>(ceil_div(n, 256), (int64_t)cus * 32);
    k_sample_short<<<(unsigned)std::max<int64_t>(1, grid_short), 256, 0, s>>>(csc.in_off, csc.in_src, n, k, o,
                                                                             rank_list, rank_count);
    TAURUS_CHECK_LAUNCH();
    if (k < LIGHT_MAX) {  // else every list of at most LIGHT_MAX in-edges is kept whole
        k_sample_light<<<(unsigned)cus * 32, 256, 0, s>>>(csc.in_off, csc.in_src, rank_list, rank_count, seed, layer,
                                                          k, o);
        TAURUS_CHECK_LAUNCH();
    }
    if (csc.nheavy > 0) {
        if (k <= HEAVY_SMALL_K) {
            const int64_t grid = std::min<int64_t>(ceil_div(csc.nheavy, 4), (int64_t)cus * 32);
            k_sample_heavy<HEAVY_CAP_SMALL><<<(unsigned)grid, 256, 0, s>>>(csc.in_off, csc.in_src, csc.heavy,
                                                                          csc.nheavy, seed, layer, k, o);
        } else {
            const int64_t grid = std::min<int64_t>(ceil_div(csc.nheavy, 4), (int64_t)cus * 12);
            k_sample_heavy<HEAVY_CAP><<<(unsigned)grid, 256, 0, s>>>(csc.in_off, csc.in_src, csc.heavy, csc.nheavy,
                                                                    seed, layer, k, o);
        }
        TAURUS_CHECK_LAUNCH();
    }
}

// kept per destination, min(d_in(v), k)
__global__ void k_sample_counts(const int64_t* __restrict__ in_off, int64_t n, int k, int32_t* __restrict__ m) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n) m[v] = (int32_t)min(in_off[v + 1] - in_off[v], (int64_t)k);
}

int64_t sample_items(const Csc& csc, int64_t n, uint64_t seed, int layer, int k, int64_t C, int vbits,
                     Arena& key_arena, Arena& val_arena, SortBuffers& sb, int32_t* m, int32_t* first_chunk, int* bad,
                     hipStream_t s) {
    if (k < 1 || k > FANOUT_MAX) fail(TAURUS_E_INVALID, "fanout %d outside [1, %d]", k, FANOUT_MAX);
    int64_t* koff = key_arena.alloc<int64_t>(n + 1, "kept before each destination");
    k_sample_counts<<<(unsigned)ceil_div(n, 256), 256, 0, s>>>(csc.in_off, n, k, m);
    TAURUS_CHECK_LAUNCH();
    scan_i32_to_i64(m, koff, n, true, key_arena, s);
    int64_t kept = 0;
    {
        Readback rb;
        rb.add(&kept, koff + n, 1);
        rb.run(s);
    }
    const int64_t k1 = std::max<int64_t>(kept, 1);
    sb.keys[0] = key_arena.alloc<uint64_t>(k1, "index keys");
    sb.keys[1] = key_arena.alloc<uint64_t>(k1, "index keys (ping-pong)");
    sb.vals[0] = val_arena.alloc<uint32_t>(k1, "index values");
    sb.vals[1] = val_arena.alloc<uint32_t>(k1, "index values (ping-pong)");
    sb.cur = 0;
    if (kept > 0)
        sample_pass(csc, n, seed, layer, k,
                    SampleOut{sb.keys[0], sb.vals[0], koff, C, vbits, nullptr, nullptr, nullptr, bad, first_chunk},
                    key_arena, s);
    return kept;
}

void sample_mask(const taurus_graph& g, const Csc& csc, uint64_t seed, int layer, int k, uint64_t* mask,
                 hipStream_t s) {
    const int64_t words = ceil_div(g.e, 64);
    if (words == 0) return;
    fill_i32(reinterpret_cast<int32_t*>(mask), 2 * words, 0, s);
    Arena tmp(s);
    int* bad = tmp.alloc<int>(1, "sampler flag");
    fill_i32(bad, 1, 0, s);
    sample_pass(csc, g.n, seed, layer, k,
                SampleOut{nullptr, nullptr, nullptr, 1, 1, reinterpret_cast<unsigned long long*>(mask), g.row_off,
                          g.col_dst, bad, nullptr},
                tmp, s);
    int hbad = 0;
    Readback rb;
    rb.add(&hbad, bad, 1);
    rb.run(s);
    if (hbad) fail(TAURUS_E_INVALID, "sampler: an in-list holds repeated sources");
}

}  // namespace taurus
