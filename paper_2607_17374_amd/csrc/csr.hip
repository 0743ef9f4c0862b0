// CSR by source (Sec. 3.2: topology is stored as CSR over out-edges so that
// sources are scanned in vertex order).  Built by a stable radix sort of the
// (u, v) pairs packed into 64-bit keys; row offsets come from a binary search
// of each row's first key in the sorted array.
#include "internal.hpp"

namespace taurus {

// pack (u, v) into u << vbits | v and flag out-of-range ids and self loops.
// Workgroup t packs tile t of RADIX_TILE edges and counts the low 8 bits of
// its keys, the radix sort's first digit: hist[digit * tiles + t].
__global__ __launch_bounds__(256) void k_pack_edges(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                                                    int64_t e, int64_t n, int vbits, uint64_t* __restrict__ keys,
                                                    int* __restrict__ bad, uint32_t* __restrict__ hist,
                                                    int64_t tiles) {
    __shared__ uint32_t h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * RADIX_TILE;
    bool flag = false;
    for (int j = 0; j < RADIX_TILE / 256; j++) {
        const int64_t i = base + (int64_t)j * 256 + threadIdx.x;
        if (i >= e) break;
        const int64_t u = src[i], v = dst[i];
        uint64_t key = 0;
        if (u < 0 || u >= n || v < 0 || v >= n || u == v) flag = true;
        else key = ((uint64_t)u << vbits) | (uint64_t)v;
        keys[i] = key;
        atomicAdd(&h[key & 255u], 1u);
    }
    if (flag) atomicOr(bad, 1);
    __syncthreads();
    hist[(int64_t)threadIdx.x * tiles + blockIdx.x] = h[threadIdx.x];
}

// col_dst from the sorted keys; a key equal to its predecessor is a repeat
__global__ void k_unpack_cols(const uint64_t* __restrict__ keys, int64_t e, int vbits,
                              int32_t* __restrict__ col_dst, int* __restrict__ bad) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= e) return;
    const uint64_t k = keys[i];
    col_dst[i] = (int32_t)(k & (((uint64_t)1 << vbits) - 1));
    if (i > 0 && keys[i - 1] == k) atomicOr(bad, 2);
}

// row_off[u] = first position whose source is >= u (binary search), u in [0, n]
__global__ void k_row_offsets(const uint64_t* __restrict__ keys, int64_t e, int64_t n, int vbits,
                              int64_t* __restrict__ row_off) {
    const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (u > n) return;
    const uint64_t target = (uint64_t)u << vbits;
    int64_t lo = 0, hi = e;
    while (lo < hi) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (keys[mid] < target) lo = mid + 1;
        else hi = mid;
    }
    row_off[u] = lo;
}

int build_csr_impl(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                   int32_t* col_dst, hipStream_t s) {
    if (n <= 0 || n >= ((int64_t)1 << 31) || e < 0 || e >= ((int64_t)1 << 40))
        fail(TAURUS_E_INVALID, "taurus_build_csr: n=%lld e=%lld out of range", (long long)n, (long long)e);
    if (!row_off || (e > 0 && (!src || !dst || !col_dst)))
        fail(TAURUS_E_INVALID, "taurus_build_csr: null pointer");
    Arena arena(s);
    const int vbits = bits_for(n - 1) > 0 ? bits_for(n - 1) : 1;
    int* bad = arena.alloc<int>(1, "flag");
    fill_i32(bad, 1, 0, s);
    SortBuffers sb{{arena.alloc<uint64_t>(e > 0 ? e : 1, "edge keys"), nullptr}, {nullptr, nullptr}, 0};
    const int T = 256;
    if (e > 0) {
        sb.keys[1] = arena.alloc<uint64_t>(e, "edge keys (ping-pong)");
        const int64_t tiles = ceil_div(e, RADIX_TILE);
        uint32_t* hist0 = arena.alloc<uint32_t>(256 * tiles, "first-digit histogram");
        k_pack_edges<<<(unsigned)tiles, 256, 0, s>>>(src, dst, e, n, vbits, sb.keys[0], bad, hist0, tiles);
        TAURUS_CHECK_LAUNCH();
        radix_sort_u64(sb, e, 2 * vbits, arena, s, bad, 4, hist0);
        k_unpack_cols<<<(unsigned)ceil_div(e, T), T, 0, s>>>(sb.keys[sb.cur], e, vbits, col_dst, bad);
        TAURUS_CHECK_LAUNCH();
    }
    k_row_offsets<<<(unsigned)ceil_div(n + 1, T), T, 0, s>>>(sb.keys[sb.cur], e, n, vbits, row_off);
    TAURUS_CHECK_LAUNCH();
    int hbad = 0;
    Readback rb;
    rb.add(&hbad, bad, 1);
    rb.run(s);
    if (hbad & 1) fail(TAURUS_E_INVALID, "taurus_build_csr: vertex id out of range or self loop");
    if (hbad & 2) fail(TAURUS_E_INVALID, "taurus_build_csr: repeated edge");
    if (hbad & 4) fail(TAURUS_E_DEVICE, "taurus_build_csr: radix sort offset out of range");
    return TAURUS_OK;
}

}  // namespace taurus
