// Fanout sampling (Sec. 3.9, "Sampling-based Inference"): for every
// destination v keep the min(d_in(v), k) in-edges (u, v) whose rank pairs
// (H(seed, 4, layer, v, u), u) are smallest; the rest do not propagate in
// this layer.
//
// The in-edges of each destination are read from a CSC, built once per
// graph by a stable radix sort of the CSR edges by destination (sources stay
// ascending within a destination).  Then, per layer:
//   1. threshold: for every v with d_in(v) > k a wave finds tau_v, the k-th
//      smallest rank pair of its in-edges.  The wave takes the in-edges 64
//      at a time, sorts each batch across its lanes (bitonic network on
//      (key, u) pairs) and merges it into a running sorted list of the 64
//      smallest pairs so far; a batch with no pair below the running k-th
//      smallest is skipped without sorting.  Destinations with more than
//      512 in-edges are cut into pieces taken by separate waves, whose
//      k smallest pairs are merged when the last piece is done, so a hub
//      costs no more wall time than a piece;
//   2. mask: one pass over the CSR in edge order keeps (u, v) iff its pair is
//      <= tau_v (tau_v = +inf when d_in(v) <= k); each wave's 64 decisions
//      form one mask word by ballot, so no atomics are needed.
// Rank pairs are distinct within a destination (the sources are), so the
// kept set is unique and the mask is exact.
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

// CSR edge i -> sort key v, value u
__global__ __launch_bounds__(256) void k_csc_items(const int64_t* __restrict__ row_off,
                                                   const int32_t* __restrict__ col_dst, int64_t n, int64_t e,
                                                   uint64_t* __restrict__ keys, uint32_t* __restrict__ vals) {
    __shared__ int64_t ro[4][64];
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t u = wave_edge_row(row_off, n, i, ro[threadIdx.x >> 6]);
    if (i >= e) return;
    keys[i] = (uint64_t)col_dst[i];
    vals[i] = (uint32_t)u;
}

// in_off[v] = first position of the sorted destinations that is >= v
// (binary search; no atomics, so hubs cost nothing extra), v in [0, n]
__global__ void k_csc_offsets(const uint64_t* __restrict__ keys, int64_t e, int64_t n, int64_t* __restrict__ in_off) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v > n) return;
    int64_t lo = 0, hi = e;
    while (lo < hi) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (keys[mid] < (uint64_t)v) lo = mid + 1;
        else hi = mid;
    }
    in_off[v] = lo;
}

std::shared_ptr<Csc> build_csc(const taurus_graph& g, hipStream_t s) {
    const auto t0 = std::chrono::steady_clock::now();
    auto c = std::make_shared<Csc>(s);
    const int64_t n = g.n, e = g.e;
    const int T = 256;
    validate_csr(g, s);
    Arena tmp(s);
    int* bad = tmp.alloc<int>(1, "sort flag");
    fill_i32(bad, 1, 0, s);
    int hbad = 0;
    c->in_off = c->arena.alloc<int64_t>(n + 1, "in-edge offsets");
    if (e > 0) {
        SortBuffers sb{{tmp.alloc<uint64_t>(e, "csc keys"), tmp.alloc<uint64_t>(e, "csc keys (ping-pong)")},
                       {c->arena.alloc<uint32_t>(e, "in-edge sources"),
                        c->arena.alloc<uint32_t>(e, "in-edge sources (ping-pong)")},
                       0};
        k_csc_items<<<(unsigned)ceil_div(e, T), T, 0, s>>>(g.row_off, g.col_dst, n, e, sb.keys[0], sb.vals[0]);
        TAURUS_CHECK_LAUNCH();
        radix_sort_u64(sb, e, std::max(1, bits_for(n - 1)), tmp, s, bad, 8);
        c->in_src = reinterpret_cast<int32_t*>(sb.vals[sb.cur]);
        c->arena.free_ptr(sb.vals[1 - sb.cur]);
        k_csc_offsets<<<(unsigned)ceil_div(n + 1, T), T, 0, s>>>(sb.keys[sb.cur], e, n, c->in_off);
        TAURUS_CHECK_LAUNCH();
    } else {
        fill_i32(reinterpret_cast<int32_t*>(c->in_off), 2 * (n + 1), 0, s);
    }
    {
        Readback rb;
        rb.add(&hbad, bad, 1);
        rb.run(s);
    }
    if (hbad) fail(TAURUS_E_DEVICE, "in-edge sort: radix offset out of range");
    c->ms_build = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    return c;
}

// ------------------------------------------------------------- threshold ----
__device__ inline bool pair_less(uint64_t ka, uint32_t ua, uint64_t kb, uint32_t ub) {
    return ka < kb || (ka == kb && ua < ub);
}

__device__ inline uint64_t shfl64(uint64_t x, int src) {
    const uint32_t lo = __shfl((uint32_t)x, src, 64), hi = __shfl((uint32_t)(x >> 32), src, 64);
    return ((uint64_t)hi << 32) | lo;
}

// Compare-exchange with lane ^ stride: keep the smaller pair if keep_min.
__device__ inline void exchange(uint64_t& k, uint32_t& u, int stride, bool keep_min) {
    const int lane = threadIdx.x & 63;
    const uint64_t pk = shfl64(k, lane ^ stride);
    const uint32_t pu = __shfl(u, lane ^ stride, 64);
    const bool p_less = pair_less(pk, pu, k, u);
    if (keep_min == p_less) {
        k = pk;
        u = pu;
    }
}

// Sort the wave's 64 pairs ascending by lane (bitonic network).
__device__ inline void bitonic_sort64(uint64_t& k, uint32_t& u) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int size = 2; size <= 64; size <<= 1)
#pragma unroll
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            const bool ascending = (lane & size) == 0 || size == 64;
            const bool lower = (lane & stride) == 0;
            exchange(k, u, stride, lower == ascending);
        }
}

// (ck, cu) ascending and (bk, bu) ascending -> the 64 smallest of both,
// ascending: lane-wise minimum against the reversed batch is bitonic, and a
// bitonic merge sorts it.
__device__ inline void merge_smallest(uint64_t& ck, uint32_t& cu, uint64_t bk, uint32_t bu) {
    const int lane = threadIdx.x & 63;
    const uint64_t rk = shfl64(bk, 63 - lane);
    const uint32_t ru = __shfl(bu, 63 - lane, 64);
    if (pair_less(rk, ru, ck, cu)) {
        ck = rk;
        cu = ru;
    }
#pragma unroll
    for (int stride = 32; stride > 0; stride >>= 1) exchange(ck, cu, stride, (lane & stride) == 0);
}

constexpr int SAMPLE_BATCHES = 8;
// destinations with more in-edges than this are split into pieces of as many
// in-edges (k_sample_pieces); the others are scanned whole (k_sample_threshold)
constexpr int64_t SAMPLE_PIECE = 64 * SAMPLE_BATCHES;

// The 64 smallest rank pairs among v's in-edges [a, b) merged into the
// wave's running list (ck, cu), ascending by lane; pre = v's hash prefix.
// SAMPLE_BATCHES batches of 64 in-edges are loaded at a time, so a long scan
// keeps that many loads in flight; a batch with no pair below the running
// k-th smallest is skipped without sorting.
__device__ inline void scan_smallest(const int32_t* __restrict__ in_src, int64_t a, int64_t b, uint64_t pre, int k,
                                     uint64_t& ck, uint32_t& cu) {
    const int lane = threadIdx.x & 63;
    for (int64_t base = a; base < b; base += 64 * SAMPLE_BATCHES) {
        // past the end a lane holds (~0, ~0), which is never below a running
        // pair and sorts last
        uint32_t uu[SAMPLE_BATCHES];
#pragma unroll
        for (int t = 0; t < SAMPLE_BATCHES; t++) {
            const int64_t idx = base + t * 64 + lane;
            uu[t] = idx < b ? (uint32_t)in_src[idx] : ~0u;
        }
#pragma unroll
        for (int t = 0; t < SAMPLE_BATCHES; t++) {
            if (base + t * 64 >= b) break;  // uniform over the wave
            const bool valid = base + t * 64 + lane < b;
            uint32_t u = uu[t];
            uint64_t key = valid ? sample_key(pre, u) : ~0ull;
            const uint64_t tk = shfl64(ck, k - 1);
            const uint32_t tu = __shfl(cu, k - 1, 64);
            if (__ballot(valid && pair_less(key, u, tk, tu)) == 0) continue;
            bitonic_sort64(key, u);
            merge_smallest(ck, cu, key, u);
        }
    }
}

// destinations per wave of k_sample_threshold: few, so that a run of
// mid-degree destinations (natural RMAT IDs cluster them) is spread over
// many waves
constexpr int SAMPLE_DPW = 8;

// One wave per SAMPLE_DPW consecutive destinations; those with k < d_in <=
// SAMPLE_PIECE are scanned one after another by the whole wave.
__global__ __launch_bounds__(256) void k_sample_threshold(const int64_t* __restrict__ in_off,
                                                          const int32_t* __restrict__ in_src, int64_t n,
                                                          uint64_t seed, int layer, int k,
                                                          uint64_t* __restrict__ thr_key,
                                                          uint32_t* __restrict__ thr_u) {
    const int lane = threadIdx.x & 63;
    const int64_t v0 = (((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6) * SAMPLE_DPW;
    if (v0 >= n) return;  // uniform over the wave
    const int64_t myv = v0 + lane;
    int64_t b = 0, d = 0;
    if (lane < SAMPLE_DPW && myv < n) {
        b = in_off[myv];
        d = in_off[myv + 1] - b;
        if (d <= k) {  // every in-edge is kept
            thr_key[myv] = ~0ull;
            thr_u[myv] = ~0u;
        }
    }
    uint64_t todo = __ballot(lane < SAMPLE_DPW && myv < n && d > k && d <= SAMPLE_PIECE);
    while (todo) {
        const int j = __ffsll((unsigned long long)todo) - 1;
        todo &= todo - 1;
        const int64_t v = v0 + j;
        const int64_t vb = (int64_t)shfl64((uint64_t)b, j), vd = (int64_t)shfl64((uint64_t)d, j);
        uint64_t ck = ~0ull;
        uint32_t cu = ~0u;
        scan_smallest(in_src, vb, vb + vd, sample_prefix(seed, (uint64_t)layer, (uint64_t)v), k, ck, cu);
        if (lane == k - 1) {
            thr_key[v] = ck;
            thr_u[v] = cu;
        }
    }
}

// The destination whose in-edges hold CSC position pos (0 <= pos < e): the
// largest v with in_off[v] <= pos, found by the whole wave (every lane with
// the same pos) with a 64-ary search: each round the lanes probe 64 evenly
// spaced offsets, and since in_off is non-decreasing the probes that pass
// form a prefix of the lanes.
__device__ inline int64_t covering(const int64_t* __restrict__ in_off, int64_t n, int64_t pos) {
    const int lane = threadIdx.x & 63;
    int64_t lo = 0, hi = n - 1;  // the answer lies in [lo, hi]
    while (hi - lo >= 64) {
        const int64_t step = (hi - lo + 63) / 64;
        const int64_t q = min(lo + (int64_t)(lane + 1) * step, hi);
        const int c = __popcll(__ballot(in_off[q] <= pos));
        const int64_t nhi = min(hi, lo + (int64_t)(c + 1) * step - 1);
        lo = min(lo + (int64_t)c * step, hi);
        hi = nhi;
    }
    const bool ok = lo + lane <= hi && in_off[lo + lane] <= pos;
    return lo + __popcll(__ballot(ok)) - 1;
}

// Destinations with more than SAMPLE_PIECE in-edges.  One wave per piece of
// SAMPLE_PIECE consecutive CSC positions.  A piece meets at most two such
// destinations: the one holding its first position (slot 0) and one starting
// inside it, which then holds its last position (slot 1).  For each, the
// wave writes the k smallest pairs of its part of the piece to
// piece_key/piece_u[(p * 2 + slot) * k + i]; the last piece of a destination
// to finish (a counter per destination, behind a device-scope fence) merges
// the destination's pieces in order and writes its threshold.
__global__ __launch_bounds__(256) void k_sample_pieces(const int64_t* __restrict__ in_off,
                                                       const int32_t* __restrict__ in_src, int64_t n, int64_t e,
                                                       uint64_t seed, int layer, int k,
                                                       uint64_t* __restrict__ piece_key,
                                                       uint32_t* __restrict__ piece_u, int32_t* __restrict__ done,
                                                       uint64_t* __restrict__ thr_key,
                                                       uint32_t* __restrict__ thr_u) {
    const int lane = threadIdx.x & 63;
    const int64_t p = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (p >= (e + SAMPLE_PIECE - 1) / SAMPLE_PIECE) return;  // uniform over the wave
    const int64_t start = p * SAMPLE_PIECE, end = min(e, start + SAMPLE_PIECE);
    const int64_t va = covering(in_off, n, start), vz = covering(in_off, n, end - 1);
    for (int slot = 0; slot < 2; slot++) {
        if (slot == 1 && vz == va) break;
        const int64_t v = slot == 0 ? va : vz;
        const int64_t vb = in_off[v], ve = in_off[v + 1];
        if (ve - vb <= SAMPLE_PIECE) continue;
        const uint64_t pre = sample_prefix(seed, (uint64_t)layer, (uint64_t)v);
        uint64_t ck = ~0ull;
        uint32_t cu = ~0u;
        scan_smallest(in_src, max(vb, start), min(ve, end), pre, k, ck, cu);
        const int64_t r = (p * 2 + slot) * k;
        if (lane < k) {
            piece_key[r + lane] = ck;
            piece_u[r + lane] = cu;
        }
        __threadfence();
        const int64_t p0 = vb / SAMPLE_PIECE, p1 = (ve - 1) / SAMPLE_PIECE;
        int last = 0;
        if (lane == 0) last = atomicAdd(&done[v], 1) == (int)(p1 - p0) ? 1 : 0;
        if (__shfl(last, 0, 64) == 0) continue;
        __threadfence();
        ck = ~0ull;
        cu = ~0u;
        for (int64_t q = p0; q <= p1; q++) {
            // v holds the first position of every piece but possibly p0
            const int64_t rq = (q * 2 + ((q == p0 && vb != q * SAMPLE_PIECE) ? 1 : 0)) * k;
            const uint64_t bk = lane < k ? piece_key[rq + lane] : ~0ull;
            const uint32_t bu = lane < k ? piece_u[rq + lane] : ~0u;
            merge_smallest(ck, cu, bk, bu);
        }
        if (lane == k - 1) {
            thr_key[v] = ck;
            thr_u[v] = cu;
        }
    }
}

// ------------------------------------------------------------------ mask ----
__global__ __launch_bounds__(256) void k_sample_mask(const int64_t* __restrict__ row_off,
                                                     const int32_t* __restrict__ col_dst, int64_t n, int64_t e,
                                                     uint64_t seed, int layer,
                                                     const uint64_t* __restrict__ thr_key,
                                                     const uint32_t* __restrict__ thr_u,
                                                     uint64_t* __restrict__ mask) {
    __shared__ int64_t ro[4][64];
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int lane = threadIdx.x & 63;
    const int64_t u = wave_edge_row(row_off, n, i, ro[threadIdx.x >> 6]);
    bool keep = false;
    if (i < e) {
        const int32_t v = col_dst[i];
        const uint64_t key = sample_key(sample_prefix(seed, (uint64_t)layer, (uint64_t)v), (uint64_t)u);
        keep = !pair_less(thr_key[v], thr_u[v], key, (uint32_t)u);
    }
    const uint64_t word = __ballot(keep);
    const int64_t i0 = i - lane;
    if (lane == 0 && i0 < e) mask[i0 >> 6] = word;
}

void sample_mask(const taurus_graph& g, const Csc& csc, uint64_t seed, int layer, int k, uint64_t* mask,
                 hipStream_t s) {
    const int64_t n = g.n, e = g.e;
    if (e == 0) return;
    if (k < 1 || k > 64) fail(TAURUS_E_INVALID, "fanout %d outside [1, 64]", k);
    Arena tmp(s);
    uint64_t* thr_key = tmp.alloc<uint64_t>(n, "sampling thresholds");
    uint32_t* thr_u = tmp.alloc<uint32_t>(n, "sampling thresholds (sources)");
    const int64_t pieces = ceil_div(e, SAMPLE_PIECE);
    uint64_t* piece_key = tmp.alloc<uint64_t>(pieces * 2 * k, "piece pairs");
    uint32_t* piece_u = tmp.alloc<uint32_t>(pieces * 2 * k, "piece pairs (sources)");
    int32_t* done = tmp.alloc<int32_t>(n, "pieces done");
    fill_i32(done, n, 0, s);
    k_sample_pieces<<<(unsigned)ceil_div(pieces, 4), 256, 0, s>>>(csc.in_off, csc.in_src, n, e, seed, layer, k,
                                                                 piece_key, piece_u, done, thr_key, thr_u);
    TAURUS_CHECK_LAUNCH();
    const int64_t waves = ceil_div(n, SAMPLE_DPW);
    k_sample_threshold<<<(unsigned)ceil_div(waves, 4), 256, 0, s>>>(csc.in_off, csc.in_src, n, seed, layer, k, thr_key,
                                                                   thr_u);
    TAURUS_CHECK_LAUNCH();
    k_sample_mask<<<(unsigned)ceil_div(e, 256), 256, 0, s>>>(g.row_off, g.col_dst, n, e, seed, layer, thr_key, thr_u,
                                                            mask);
    TAURUS_CHECK_LAUNCH();
}

}  // namespace taurus
