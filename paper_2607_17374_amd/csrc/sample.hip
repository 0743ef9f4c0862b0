// Fanout sampling (Sec. 3.9, "Sampling-based Inference"): for every
// destination v keep the min(d_in(v), k) in-edges (u, v) whose rank pairs
// (H(seed, 4, layer, v, u), u) are smallest; the rest do not propagate in
// this layer.
//
// The in-edges of each destination are read from a CSC, built once per
// graph by a stable radix sort of the CSR edges by destination (sources stay
// ascending within a destination).  Then, per layer:
//   1. threshold: for every v with d_in(v) > k one wave finds tau_v, the k-th
//      smallest rank pair of its in-edges.  The wave takes the in-edges 64
//      at a time, sorts each batch across its lanes (bitonic network on
//      (key, u) pairs) and merges it into a running sorted list of the 64
//      smallest pairs so far; a batch with no pair below the running k-th
//      smallest is skipped without sorting, so hubs cost little more than a
//      pass over their keys;
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

// CSR edge i -> sort key v, value u; in-degree counts
__global__ __launch_bounds__(256) void k_csc_items(const int64_t* __restrict__ row_off,
                                                   const int32_t* __restrict__ col_dst, int64_t n, int64_t e,
                                                   uint64_t* __restrict__ keys, uint32_t* __restrict__ vals,
                                                   int32_t* __restrict__ deg) {
    __shared__ int64_t ro[4][64];
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t u = wave_edge_row(row_off, n, i, ro[threadIdx.x >> 6]);
    if (i >= e) return;
    const int32_t v = col_dst[i];
    keys[i] = (uint64_t)v;
    vals[i] = (uint32_t)u;
    atomicAdd(&deg[v], 1);
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
    int32_t* deg = tmp.alloc<int32_t>(n, "in-degrees");
    fill_i32(deg, n, 0, s);
    c->in_off = c->arena.alloc<int64_t>(n + 1, "in-edge offsets");
    if (e > 0) {
        SortBuffers sb{{tmp.alloc<uint64_t>(e, "csc keys"), tmp.alloc<uint64_t>(e, "csc keys (ping-pong)")},
                       {c->arena.alloc<uint32_t>(e, "in-edge sources"),
                        c->arena.alloc<uint32_t>(e, "in-edge sources (ping-pong)")},
                       0};
        k_csc_items<<<(unsigned)ceil_div(e, T), T, 0, s>>>(g.row_off, g.col_dst, n, e, sb.keys[0], sb.vals[0], deg);
        TAURUS_CHECK_LAUNCH();
        radix_sort_u64(sb, e, std::max(1, bits_for(n - 1)), tmp, s, bad, 8);
        c->in_src = reinterpret_cast<int32_t*>(sb.vals[sb.cur]);
        c->arena.free_ptr(sb.vals[1 - sb.cur]);
    }
    scan_i32_to_i64(deg, c->in_off, n, true, tmp, s);
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

// One wave per 64 consecutive destinations; destinations with more than k
// in-edges are processed one after another by the whole wave.
__global__ __launch_bounds__(256) void k_sample_threshold(const int64_t* __restrict__ in_off,
                                                          const int32_t* __restrict__ in_src, int64_t n,
                                                          uint64_t seed, int layer, int k,
                                                          uint64_t* __restrict__ thr_key,
                                                          uint32_t* __restrict__ thr_u) {
    const int lane = threadIdx.x & 63;
    const int64_t v0 = (((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6) << 6;
    if (v0 >= n) return;  // uniform over the wave
    const int64_t myv = v0 + lane;
    int64_t b = 0, d = 0;
    if (myv < n) {
        b = in_off[myv];
        d = in_off[myv + 1] - b;
        if (d <= k) {  // every in-edge is kept
            thr_key[myv] = ~0ull;
            thr_u[myv] = ~0u;
        }
    }
    uint64_t todo = __ballot(myv < n && d > k);
    while (todo) {
        const int j = __ffsll((unsigned long long)todo) - 1;
        todo &= todo - 1;
        const int64_t v = v0 + j;
        const int64_t vb = (int64_t)shfl64((uint64_t)b, j), vd = (int64_t)shfl64((uint64_t)d, j);
        const uint64_t pre = sample_prefix(seed, (uint64_t)layer, (uint64_t)v);
        uint64_t ck = ~0ull;
        uint32_t cu = ~0u;
        for (int64_t base = 0; base < vd; base += 64) {
            const bool valid = base + lane < vd;
            uint32_t u = valid ? (uint32_t)in_src[vb + base + lane] : ~0u;
            uint64_t key = valid ? sample_key(pre, u) : ~0ull;
            const uint64_t tk = shfl64(ck, k - 1);
            const uint32_t tu = __shfl(cu, k - 1, 64);
            if (__ballot(valid && pair_less(key, u, tk, tu)) == 0) continue;
            bitonic_sort64(key, u);
            merge_smallest(ck, cu, key, u);
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
    const int64_t waves = ceil_div(n, 64);
    k_sample_threshold<<<(unsigned)ceil_div(waves, 4), 256, 0, s>>>(csc.in_off, csc.in_src, n, seed, layer, k, thr_key,
                                                                   thr_u);
    TAURUS_CHECK_LAUNCH();
    k_sample_mask<<<(unsigned)ceil_div(e, 256), 256, 0, s>>>(g.row_off, g.col_dst, n, e, seed, layer, thr_key, thr_u,
                                                            mask);
    TAURUS_CHECK_LAUNCH();
}

}  // namespace taurus
