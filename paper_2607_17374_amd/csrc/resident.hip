// Accumulator residency under a device-memory budget (Sec. 3.5: a GPU
// store keeps the accumulators of high in-degree hub vertices resident; the
// partial states of other destinations live in a bounded pool and, when the
// pool runs short, victims are evicted to host memory and reloaded before
// their next message).  The paper's policy evicts those with the fewest
// pending messages (Sec. 3.5.3); random, first-in-first-out and
// least-recently-used choices are its comparison policies (Sec. 4).
//
// Accumulator rows live in a pool of S slots; slot_of[v] names v's row (or
// -1).  Hubs -- the top hub_fraction of vertices by (message count
// descending, ID ascending) -- own slots 0..H-1 for the whole layer.  Before
// chunk k runs:
//   1. every destination the chunk touches (its work units and its own
//      vertices, for the self message) is marked with k; those still pending
//      and without a slot are listed;
//   2. if the free slots do not cover the list, victims are chosen among
//      resident, non-hub, still-pending vertices the chunk does not touch,
//      smallest policy key first, then lowest ID.  Keys:
//        fewest pending: the exact count of pending messages;
//        random:         the top 14 bits of H(seed, 7, k, v);
//        FIFO:           the chunk at which v last took a row;
//        LRU:            the last chunk that sent v a message.
//      A 16,384-bin histogram gives the threshold bin: pending counts of
//      16,383 and more share the last bin, and chunk numbers are shifted
//      right until the layer's chunk count fits 14 bits.  Candidates of a
//      threshold bin that holds one key value are ranked by an exclusive
//      scan in vertex order; those of a bin that holds several (the last
//      pending bin, any shifted chunk bin) are sorted by (exact key, ID).
//      The key only decides which rows move, never the results;
//      their rows are written to the pinned host store and their slots freed;
//   3. listed vertices take free slots; evicted ones copy their row back.
// After the chunk, touched vertices that completed return their slots.
// Rows are moved by exact copies, so results equal the in-core run's.
#include "device.hpp"
#include "internal.hpp"
#include "resident.hpp"

namespace taurus {

constexpr int RES_BINS = 16384;

// chunk work: items are the units of the chunk's lists, then its own rows
__device__ inline int dest_of(const ResChunk& c, int64_t t) {
#pragma unroll
    for (int l = 0; l < RES_LISTS; l++) {
        if (t < c.n[l]) return c.u[l][t].z;
        t -= c.n[l];
    }
    return (int)(c.first_row + t);
}

__global__ void k_res_collect(ResChunk c, int64_t total, int32_t k, const int32_t* __restrict__ slot_of,
                              const int2* __restrict__ cnt, int32_t* __restrict__ dc_mark,
                              int32_t* __restrict__ want, int32_t* __restrict__ need,
                              unsigned long long* __restrict__ need_count) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= total) return;
    const int v = dest_of(c, t);
    dc_mark[v] = k;
    const bool add = slot_of[v] < 0 && cnt[v].x > 0 && atomicExch(&want[v], 1) == 0;
    const unsigned long long at = wave_append(add, need_count);
    if (add) need[at] = v;
}

__device__ inline bool res_candidate(int v, int32_t k, const int32_t* slot_of, const uint8_t* hub,
                                     const int32_t* dc_mark, const int2* cnt) {
    return slot_of[v] >= 0 && !hub[v] && dc_mark[v] != k && cnt[v].x > 0;
}

// What the eviction key of a candidate reads.
struct EvictKeys {
    int policy;     // TAURUS_EVICT_*
    int shift;      // chunk numbers >> shift fit the bins
    uint64_t seed;  // random policy
    const int2* cnt;
    const int32_t* dc_mark;  // last chunk that touched v
    const int32_t* adm;      // chunk at which v last took a row
};

// the exact key a coarse bin is refined by
__device__ inline int64_t res_exact_key(int v, const EvictKeys& e) {
    switch (e.policy) {
        case TAURUS_EVICT_FIFO: return max(e.adm[v], 0);
        case TAURUS_EVICT_LRU: return max(e.dc_mark[v], 0);
        default: return max(e.cnt[v].x, 0);
    }
}

__device__ inline int res_key(int v, int32_t k, const EvictKeys& e) {
    switch (e.policy) {
        case TAURUS_EVICT_RANDOM: {
            uint64_t h = mix64(e.seed + SM64_GAMMA + 7u);
            h = mix64(h + SM64_GAMMA + (uint64_t)k);
            h = mix64(h + SM64_GAMMA + (uint64_t)v);
            return (int)(h >> 50);
        }
        case TAURUS_EVICT_FIFO: return min(max(e.adm[v], 0) >> e.shift, RES_BINS - 1);
        case TAURUS_EVICT_LRU: return min(max(e.dc_mark[v], 0) >> e.shift, RES_BINS - 1);
        default: return min(max(e.cnt[v].x, 0), RES_BINS - 1);
    }
}

__global__ __launch_bounds__(1024) void k_res_hist(int64_t n, int32_t k, const int32_t* __restrict__ slot_of,
                                                   const uint8_t* __restrict__ hub, EvictKeys e,
                                                   unsigned int* __restrict__ hist) {
    __shared__ unsigned int h[RES_BINS];
    for (int i = threadIdx.x; i < RES_BINS; i += blockDim.x) h[i] = 0;
    __syncthreads();
    for (int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; v < n; v += (int64_t)gridDim.x * blockDim.x)
        if (res_candidate((int)v, k, slot_of, hub, e.dc_mark, e.cnt)) atomicAdd(&h[res_key((int)v, k, e)], 1u);
    __syncthreads();
    for (int i = threadIdx.x; i < RES_BINS; i += blockDim.x)
        if (h[i]) atomicAdd(&hist[i], h[i]);
}

__global__ void k_res_tie_flags(int64_t n, int32_t k, int32_t tau, const int32_t* __restrict__ slot_of,
                                const uint8_t* __restrict__ hub, EvictKeys e, int32_t* __restrict__ tie) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n) return;
    tie[v] = res_candidate((int)v, k, slot_of, hub, e.dc_mark, e.cnt) && res_key((int)v, k, e) == tau ? 1 : 0;
}

// the candidates of a coarse threshold bin, keyed (exact key, ID)
__global__ void k_res_tie_keys(int64_t n, const int32_t* __restrict__ tie, const int64_t* __restrict__ tie_rank,
                               EvictKeys e, int idbits, uint64_t* __restrict__ keys, uint32_t* __restrict__ ids) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n || !tie[v]) return;
    const int64_t j = tie_rank[v];
    keys[j] = ((uint64_t)res_exact_key((int)v, e) << idbits) | (uint64_t)v;
    ids[j] = (uint32_t)v;
}

// the sorted position of each coarse-bin candidate becomes its tie rank
__global__ void k_res_tie_ranks(const uint32_t* __restrict__ order, int64_t m, int64_t* __restrict__ tie_rank) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j < m) tie_rank[order[j]] = j;
}

__global__ void k_res_victims(int64_t n, int32_t k, int32_t tau, int64_t tie_take,
                              const int32_t* __restrict__ slot_of, const uint8_t* __restrict__ hub, EvictKeys e,
                              const int64_t* __restrict__ tie_rank, int32_t* __restrict__ victims,
                              unsigned long long* __restrict__ count) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n || !res_candidate((int)v, k, slot_of, hub, e.dc_mark, e.cnt)) return;
    const int b = res_key((int)v, k, e);
    const bool add = b < tau || (b == tau && tie_rank[v] < tie_take);
    const unsigned long long at = wave_append(add, count);
    if (add) victims[at] = (int32_t)v;
}

// one wave per victim: row to the host store, slot back to the free list
__global__ __launch_bounds__(256) void k_res_evict(const int32_t* __restrict__ victims, int64_t nv, int d_o,
                                                   float* __restrict__ pool, float* __restrict__ store,
                                                   int32_t* __restrict__ slot_of, uint8_t* __restrict__ evicted,
                                                   int32_t* __restrict__ free_list, int32_t base) {
    const int64_t j = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    const int lane = threadIdx.x & 63;
    if (j >= nv) return;
    const int v = victims[j];
    const int32_t s = slot_of[v];
    const float4* src = reinterpret_cast<const float4*>(pool + (int64_t)s * d_o);
    float4* dst = reinterpret_cast<float4*>(store + (int64_t)v * d_o);
    for (int q = lane; q < d_o / 4; q += 64) dst[q] = src[q];
    if (lane == 0) {
        slot_of[v] = -1;
        evicted[v] = 1;
        free_list[base + j] = s;
    }
}

// one wave per listed vertex: take slot free_list[top - 1 - j] at chunk k;
// reload if evicted
// A wave per listed destination (waves stride over the list): take the
// free slot top - 1 - j, reloading the row if it was evicted.  nn and top
// come from the host (nn_dev null) or from device memory (the listed count
// and the free-list top), for a launch sized for the most the chunk can
// list.
__global__ __launch_bounds__(256) void k_res_assign(const int32_t* __restrict__ need, int64_t nn,
                                                    const unsigned long long* __restrict__ nn_dev, int d_o,
                                                    const int32_t* __restrict__ free_list, int64_t top,
                                                    const int32_t* __restrict__ top_dev, int32_t k,
                                                    float* __restrict__ pool, const float* __restrict__ store,
                                                    int32_t* __restrict__ slot_of, uint8_t* __restrict__ evicted,
                                                    int32_t* __restrict__ want, int32_t* __restrict__ adm,
                                                    int32_t* __restrict__ reloads_of,
                                                    unsigned long long* __restrict__ reloads) {
    const int lane = threadIdx.x & 63;
    if (nn_dev) {
        nn = (int64_t)*nn_dev;
        top = *top_dev;
    }
    const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
    for (int64_t j = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6; j < nn; j += nw) {  // uniform
        const int v = need[j];
        const int32_t s = free_list[top - 1 - j];
        if (evicted[v]) {
            const float4* src = reinterpret_cast<const float4*>(store + (int64_t)v * d_o);
            float4* dst = reinterpret_cast<float4*>(pool + (int64_t)s * d_o);
            for (int q = lane; q < d_o / 4; q += 64) dst[q] = src[q];
        }
        __builtin_amdgcn_wave_barrier();
        if (lane == 0) {
            if (evicted[v]) {
                evicted[v] = 0;
                reloads_of[v] += 1;
                atomicAdd(reloads, 1ull);
            }
            slot_of[v] = s;
            adm[v] = k;
            want[v] = 0;
        }
    }
}

// free-list top after a device-counted assignment: *top -= listed
__global__ void k_res_take(int32_t* __restrict__ top, const unsigned long long* __restrict__ listed) {
    *top -= (int32_t)*listed;
}

// touched vertices that completed give their slot back (hub slots stay)
__global__ void k_res_release(ResChunk c, int64_t total, const int2* __restrict__ cnt,
                              const uint8_t* __restrict__ hub, int32_t* __restrict__ slot_of,
                              int32_t* __restrict__ free_list, int32_t* __restrict__ free_top) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= total) return;
    const int v = dest_of(c, t);
    if (cnt[v].x != 0 || hub[v]) return;
    const int32_t s = atomicExch(&slot_of[v], -1);
    const int32_t at = wave_append(s >= 0, free_top);
    if (s >= 0) free_list[at] = s;
}

__global__ void k_res_set(int32_t* __restrict__ p, int32_t v) { *p = v; }

// hubs: vertices order[0..H) take slots 0..H-1; free list = H..S-1
__global__ void k_res_init(const uint32_t* __restrict__ order, int64_t H, int64_t S, int32_t* __restrict__ slot_of,
                           uint8_t* __restrict__ hub, int32_t* __restrict__ free_list) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < H) {
        const uint32_t v = order[t];
        slot_of[v] = (int32_t)t;
        hub[v] = 1;
    }
    if (t < S - H) free_list[t] = (int32_t)(H + t);
}

__global__ void k_hub_keys(const int32_t* __restrict__ m, int64_t n, int idbits, int64_t maxm,
                           uint64_t* __restrict__ keys, uint32_t* __restrict__ vals) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n) return;
    keys[v] = ((uint64_t)(maxm - m[v]) << idbits) | (uint64_t)v;
    vals[v] = (uint32_t)v;
}

__global__ void k_fill_u8(uint8_t* __restrict__ p, int64_t n, uint8_t v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void k_sum_hub_messages(const int32_t* __restrict__ m, const uint8_t* __restrict__ hub, int64_t n,
                                   unsigned long long* __restrict__ sum) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n && hub[v]) atomicAdd(sum, (unsigned long long)m[v]);
}

// histogram of per-vertex reload counts; the last bin takes the rest
__global__ void k_reload_hist(const int32_t* __restrict__ reloads_of, int64_t n, int bins,
                              unsigned long long* __restrict__ hist) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n) atomicAdd(&hist[min(reloads_of[v], bins - 1)], 1ull);
}

int64_t Residency::fixed_bytes(int64_t n) {
    // slot_of, dc_mark, want, tie flags, admission chunks, reload counts
    // (int32); tie ranks (int64); victims, need list (int32); hub, evicted
    // (u8); histogram
    return n * (4 + 4 + 4 + 4 + 4 + 4 + 8 + 4 + 4 + 1 + 1) + RES_BINS * 4 + 4096;
}

Residency::Residency(hipStream_t s, int64_t n_, int d_o_, int64_t slots, int64_t hubs, const int32_t* m,
                     int64_t messages, int policy_, uint64_t seed_, int64_t nchunks)
    : arena(s), n(n_), d_o(d_o_), S(slots), H(hubs), policy(policy_), seed(seed_) {
    const int cbits = bits_for(std::max<int64_t>(nchunks - 1, 0));
    chunk_shift = cbits > 14 ? cbits - 14 : 0;
    const int T = 256;
    const unsigned nb = (unsigned)ceil_div(n, T);
    slot_of = arena.alloc<int32_t>(n, "accumulator slots");
    dc_mark = arena.alloc<int32_t>(n, "chunk marks");
    want = arena.alloc<int32_t>(n, "slot requests");
    tie = arena.alloc<int32_t>(n, "eviction ties");
    adm = arena.alloc<int32_t>(n, "admission chunks");
    reloads_of = arena.alloc<int32_t>(n, "reloads per vertex");
    tie_rank = arena.alloc<int64_t>(n + 1, "eviction tie ranks");
    victims = arena.alloc<int32_t>(n, "eviction victims");
    need = arena.alloc<int32_t>(n, "slot list");
    hub = arena.alloc<uint8_t>(n, "hub flags");
    evicted = arena.alloc<uint8_t>(n, "evicted flags");
    hist = arena.alloc<unsigned int>(RES_BINS, "pending histogram");
    counters = arena.alloc<unsigned long long>(4, "residency counters");
    free_list = arena.alloc<int32_t>(S, "free slots");
    free_top = arena.alloc<int32_t>(1, "free slot count");
    pool = arena.alloc<float>(S * (int64_t)d_o, "accumulator pool");
    fill_i32(slot_of, n, -1, s);
    fill_i32(dc_mark, n, -1, s);
    fill_i32(want, n, 0, s);
    fill_i32(adm, n, 0, s);
    fill_i32(reloads_of, n, 0, s);
    k_fill_u8<<<nb, T, 0, s>>>(hub, n, 0);
    TAURUS_CHECK_LAUNCH();
    k_fill_u8<<<nb, T, 0, s>>>(evicted, n, 0);
    TAURUS_CHECK_LAUNCH();
    fill_i32(reinterpret_cast<int32_t*>(counters), 8, 0, s);
    // hubs: the first H vertices by (message count descending, ID ascending)
    Arena tmp(s);
    uint32_t* order = nullptr;
    if (H > 0) {
        const int idbits = std::max(1, bits_for(n - 1));
        const int mbits = std::max(1, bits_for(std::max<int64_t>(messages, 1)));
        if (idbits + mbits > 64) fail(TAURUS_E_INVALID, "hub key does not fit 64 bits");
        SortBuffers sb{{tmp.alloc<uint64_t>(n, "hub keys"), tmp.alloc<uint64_t>(n, "hub keys (ping-pong)")},
                       {tmp.alloc<uint32_t>(n, "hub order"), tmp.alloc<uint32_t>(n, "hub order (ping-pong)")},
                       0};
        int* bad = tmp.alloc<int>(1, "sort flag");
        fill_i32(bad, 1, 0, s);
        k_hub_keys<<<nb, T, 0, s>>>(m, n, idbits, messages, sb.keys[0], sb.vals[0]);
        TAURUS_CHECK_LAUNCH();
        radix_sort_u64(sb, n, idbits + mbits, tmp, s, bad, 1);
        order = sb.vals[sb.cur];
    }
    k_res_init<<<(unsigned)ceil_div(std::max<int64_t>(S, 1), T), T, 0, s>>>(order, H, S, slot_of, hub, free_list);
    TAURUS_CHECK_LAUNCH();
    k_res_set<<<1, 1, 0, s>>>(free_top, (int32_t)(S - H));
    TAURUS_CHECK_LAUNCH();
    free_lb = S - H;
    unsigned long long hub_msgs = 0;
    if (H > 0) {
        k_sum_hub_messages<<<nb, T, 0, s>>>(m, hub, n, counters + 3);
        TAURUS_CHECK_LAUNCH();
    }
    Readback rb;
    rb.add(&hub_msgs, counters + 3, 1);
    rb.run(s);
    hub_share = messages > 0 ? (double)hub_msgs / (double)messages : 0.0;
    // host store for evicted rows: pinned, written and read by kernels only
    store_host = static_cast<float*>(pinned_acquire((size_t)n * d_o * sizeof(float), &store_cap));
    TAURUS_HIP(hipHostGetDevicePointer(reinterpret_cast<void**>(&store_dev), store_host, 0));
}

Residency::~Residency() {
    (void)hipDeviceSynchronize();
    pinned_return(store_host, store_cap);
}

void Residency::prepare(const ResChunk& c, int32_t k, const int2* cnt, hipStream_t s) {
    const int T = 256;
    const int64_t total = c.total();
    unsigned long long* need_count = counters;
    fill_i32(reinterpret_cast<int32_t*>(need_count), 2, 0, s);
    k_res_collect<<<(unsigned)ceil_div(std::max<int64_t>(total, 1), T), T, 0, s>>>(c, total, k, slot_of, cnt, dc_mark,
                                                                                  want, need, need_count);
    TAURUS_CHECK_LAUNCH();
    // the chunk lists at most `total` destinations: with at least that many
    // slots surely free, assign them without a readback
    const int64_t grid_cap = 4096;  // workgroups of four waves, striding over the list
    if (total <= free_lb) {
        if (total > 0) {
            k_res_assign<<<(unsigned)std::min<int64_t>(ceil_div(total, 4), grid_cap), T, 0, s>>>(
                need, 0, need_count, d_o, free_list, 0, free_top, k, pool, store_dev, slot_of, evicted, want, adm,
                reloads_of, counters + 2);
            TAURUS_CHECK_LAUNCH();
            k_res_take<<<1, 1, 0, s>>>(free_top, need_count);
            TAURUS_CHECK_LAUNCH();
        }
        free_lb -= total;
        return;
    }
    unsigned long long nn = 0;
    int32_t top = 0;
    {
        Readback rb;
        rb.add(&nn, need_count, 1);
        rb.add(&top, free_top, 1);
        rb.run(s);
    }
    if (nn > (unsigned long long)top) {
        const int64_t M = (int64_t)nn - top;
        // threshold of the pending counts among candidates
        const EvictKeys ek{policy, chunk_shift, seed, cnt, dc_mark, adm};
        fill_i32(reinterpret_cast<int32_t*>(hist), RES_BINS, 0, s);
        k_res_hist<<<1024, 1024, 0, s>>>(n, k, slot_of, hub, ek, hist);
        TAURUS_CHECK_LAUNCH();
        std::vector<unsigned int> hh(RES_BINS);
        {
            Readback rb;
            rb.add(hh.data(), hist, RES_BINS);
            rb.run(s);
        }
        int64_t below = 0;
        int tau = -1;
        for (int b = 0; b < RES_BINS; b++) {
            if (below + hh[(size_t)b] >= M) {
                tau = b;
                break;
            }
            below += hh[(size_t)b];
        }
        if (tau < 0)
            fail(TAURUS_E_BUDGET, "accumulator pool: chunk %d needs %lld slots, only %lld can be freed", k,
                 (long long)nn, (long long)(top + below));
        k_res_tie_flags<<<(unsigned)ceil_div(n, T), T, 0, s>>>(n, k, tau, slot_of, hub, ek, tie);
        TAURUS_CHECK_LAUNCH();
        Arena tmp(s);
        scan_i32_to_i64(tie, tie_rank, n, false, tmp, s);
        // a bin holding several key values: rank its candidates by (exact key, ID)
        const bool coarse = (policy == TAURUS_EVICT_PENDING && tau == RES_BINS - 1) ||
                            ((policy == TAURUS_EVICT_FIFO || policy == TAURUS_EVICT_LRU) && chunk_shift > 0);
        const int64_t m_tie = (int64_t)hh[(size_t)tau];
        if (coarse && m_tie > 1) {
            const int idbits = std::max(1, bits_for(n - 1));
            SortBuffers sb{{tmp.alloc<uint64_t>(m_tie, "eviction tie keys"),
                            tmp.alloc<uint64_t>(m_tie, "eviction tie keys (ping-pong)")},
                           {tmp.alloc<uint32_t>(m_tie, "eviction tie order"),
                            tmp.alloc<uint32_t>(m_tie, "eviction tie order (ping-pong)")},
                           0};
            int* bad = tmp.alloc<int>(1, "sort flag");
            fill_i32(bad, 1, 0, s);
            k_res_tie_keys<<<(unsigned)ceil_div(n, T), T, 0, s>>>(n, tie, tie_rank, ek, idbits, sb.keys[0],
                                                                 sb.vals[0]);
            TAURUS_CHECK_LAUNCH();
            radix_sort_u64(sb, m_tie, 31 + idbits, tmp, s, bad, 1);
            k_res_tie_ranks<<<(unsigned)ceil_div(m_tie, T), T, 0, s>>>(sb.vals[sb.cur], m_tie, tie_rank);
            TAURUS_CHECK_LAUNCH();
        }
        unsigned long long* vcount = counters + 1;
        fill_i32(reinterpret_cast<int32_t*>(vcount), 2, 0, s);
        k_res_victims<<<(unsigned)ceil_div(n, T), T, 0, s>>>(n, k, tau, M - below, slot_of, hub, ek, tie_rank,
                                                             victims, vcount);
        TAURUS_CHECK_LAUNCH();
        unsigned long long got = 0;
        {
            Readback rb;
            rb.add(&got, vcount, 1);
            rb.run(s);
        }
        if ((int64_t)got != M)
            fail(TAURUS_E_DEVICE, "eviction chose %llu victims instead of %lld", got, (long long)M);
        k_res_evict<<<(unsigned)ceil_div(M * 64, T), T, 0, s>>>(victims, M, d_o, pool, store_dev, slot_of, evicted,
                                                              free_list, top);
        TAURUS_CHECK_LAUNCH();
        evictions += M;
        top += (int32_t)M;
    }
    if (nn > 0) {
        k_res_assign<<<(unsigned)std::min<int64_t>(ceil_div((int64_t)nn, 4), grid_cap), T, 0, s>>>(
            need, (int64_t)nn, nullptr, d_o, free_list, top, nullptr, k, pool, store_dev, slot_of, evicted, want,
            adm, reloads_of, counters + 2);
        TAURUS_CHECK_LAUNCH();
        k_res_set<<<1, 1, 0, s>>>(free_top, top - (int32_t)nn);
        TAURUS_CHECK_LAUNCH();
    }
    free_lb = (int64_t)top - (int64_t)nn;  // exact here
}

void Residency::release(const ResChunk& c, const int2* cnt, hipStream_t s) {
    const int64_t total = c.total();
    if (total == 0) return;
    k_res_release<<<(unsigned)ceil_div(total, 256), 256, 0, s>>>(c, total, cnt, hub, slot_of, free_list, free_top);
    TAURUS_CHECK_LAUNCH();
}

void Residency::reload_histogram(int64_t* counts, int bins, hipStream_t s) {
    Arena tmp(s);
    unsigned long long* h = tmp.alloc<unsigned long long>(bins, "reload histogram");
    fill_i32(reinterpret_cast<int32_t*>(h), 2 * (int64_t)bins, 0, s);
    k_reload_hist<<<(unsigned)ceil_div(std::max<int64_t>(n, 1), 256), 256, 0, s>>>(reloads_of, n, bins, h);
    TAURUS_CHECK_LAUNCH();
    std::vector<unsigned long long> hh((size_t)bins);
    Readback rb;
    rb.add(hh.data(), h, bins);
    rb.run(s);
    for (int b = 0; b < bins; b++) counts[b] = (int64_t)hh[(size_t)b];
}

int64_t Residency::reload_count(hipStream_t s) {
    unsigned long long r = 0;
    Readback rb;
    rb.add(&r, counters + 2, 1);
    rb.run(s);
    return (int64_t)r;
}

}  // namespace taurus
