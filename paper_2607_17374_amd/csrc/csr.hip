// CSR by source (Sec. 3.2: topology is stored as CSR over out-edges so that
// sources are scanned in vertex order).  Built by a stable radix sort of the
// (u, v) pairs packed into 64-bit keys; row offsets come from a binary search
// of each row's first key in the sorted array.
#include <algorithm>
#include <mutex>

#include "internal.hpp"

namespace taurus {

// pack (u, v) into u << vbits | v and flag out-of-range ids and self loops.
// Workgroup t packs tile t of RADIX_TILE edges and counts the low 8 bits of
// its keys, the radix sort's first digit: hist[t * 256 + digit].
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
    hist[(int64_t)blockIdx.x * 256 + threadIdx.x] = h[threadIdx.x];
}

// col_dst from the sorted keys; a key equal to its predecessor is a repeat.
// Also the row offsets (row_off filled with -1 beforehand): edge i is the
// first of its row u when its predecessor's row up differs, so row_off[u] =
// i, and so is every empty row between up and u when there are at most
// GAP_INLINE of them; the last edge ends the rows after it (row_off[w] = e,
// w up to n) the same way.  Longer runs of empty rows stay -1 for
// k_row_offsets_fill (a thread looping over millions of them, as after a
// relabelling that puts the vertices without out-edges last, took 0.5 s).
// Sources of the sorted keys are below n (an out-of-range id was packed as
// key 0 and flagged), so every write stays in [0, n].
constexpr int64_t GAP_INLINE = 16;
__global__ void k_unpack_cols(const uint64_t* __restrict__ keys, int64_t e, int64_t n, int vbits,
                              int32_t* __restrict__ col_dst, int64_t* __restrict__ row_off, int* __restrict__ bad) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= e) return;
    const uint64_t k = keys[i];
    col_dst[i] = (int32_t)(k & (((uint64_t)1 << vbits) - 1));
    const uint64_t kp = i > 0 ? keys[i - 1] : 0;
    if (i > 0 && kp == k) atomicOr(bad, 2);
    const int64_t u = min((int64_t)(k >> vbits), n - 1);
    const int64_t up = i > 0 ? min((int64_t)(kp >> vbits), n - 1) : -1;
    if (up < u) {
        row_off[u] = i;
        if (u - up <= GAP_INLINE)
            for (int64_t w = up + 1; w < u; w++) row_off[w] = i;
    }
    if (i == e - 1) {
        row_off[n] = e;
        if (n - u <= GAP_INLINE)
            for (int64_t w = u + 1; w < n; w++) row_off[w] = e;
    }
}

// row_off[u] = first position whose source is >= u (binary search), u in [0, n]
__device__ inline int64_t first_key_at_least(const uint64_t* __restrict__ keys, int64_t e, uint64_t target) {
    int64_t lo = 0, hi = e;
    while (lo < hi) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (keys[mid] < target) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}
__global__ void k_row_offsets(const uint64_t* __restrict__ keys, int64_t e, int64_t n, int vbits,
                              int64_t* __restrict__ row_off) {
    const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (u > n) return;
    row_off[u] = first_key_at_least(keys, e, (uint64_t)u << vbits);
}
// the rows k_unpack_cols left at -1 (long runs of empty rows)
__global__ void k_row_offsets_fill(const uint64_t* __restrict__ keys, int64_t e, int64_t n, int vbits,
                                   int64_t* __restrict__ row_off) {
    const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (u > n || row_off[u] >= 0) return;
    row_off[u] = first_key_at_least(keys, e, (uint64_t)u << vbits);
}

// Enqueues the build with every temporary from `arena`; returns the device
// flag word (bit 0: id out of range or self loop, bit 1: repeat, bit 2:
// sort inconsistency), to be read after the stream's work.
static int* enqueue_build_csr(Arena& arena, int64_t n, int64_t e, const int32_t* src, const int32_t* dst,
                              int64_t* row_off, int32_t* col_dst, hipStream_t s) {
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
        fill_i32(reinterpret_cast<int32_t*>(row_off), 2 * (n + 1), -1, s);
        k_unpack_cols<<<(unsigned)ceil_div(e, T), T, 0, s>>>(sb.keys[sb.cur], e, n, vbits, col_dst, row_off, bad);
        TAURUS_CHECK_LAUNCH();
        k_row_offsets_fill<<<(unsigned)ceil_div(n + 1, T), T, 0, s>>>(sb.keys[sb.cur], e, n, vbits, row_off);
        TAURUS_CHECK_LAUNCH();
    } else {
        k_row_offsets<<<(unsigned)ceil_div(n + 1, T), T, 0, s>>>(sb.keys[sb.cur], e, n, vbits, row_off);
        TAURUS_CHECK_LAUNCH();
    }
    return bad;
}

static void check_build_args(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                             int32_t* col_dst) {
    if (n <= 0 || n >= ((int64_t)1 << 31) || e < 0 || e >= ((int64_t)1 << 40))
        fail(TAURUS_E_INVALID, "taurus_build_csr: n=%lld e=%lld out of range", (long long)n, (long long)e);
    if (!row_off || (e > 0 && (!src || !dst || !col_dst)))
        fail(TAURUS_E_INVALID, "taurus_build_csr: null pointer");
}

static void report_build_flags(int hbad) {
    if (hbad & 1) fail(TAURUS_E_INVALID, "taurus_build_csr: vertex id out of range or self loop");
    if (hbad & 2) fail(TAURUS_E_INVALID, "taurus_build_csr: repeated edge");
    if (hbad & 4) fail(TAURUS_E_DEVICE, "taurus_build_csr: radix sort offset out of range");
}

int build_csr_impl(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                   int32_t* col_dst, hipStream_t s) {
    check_build_args(n, e, src, dst, row_off, col_dst);
    Arena arena(s);
    int* bad = enqueue_build_csr(arena, n, e, src, dst, row_off, col_dst, s);
    int hbad = 0;
    Readback rb;
    rb.add(&hbad, bad, 1);
    rb.run(s);
    report_build_flags(hbad);
    return TAURUS_OK;
}

// ---- the same build without allocating -------------------------------------
// Its temporaries live in `scratch`, one fixed array per GPU, held from the
// first call on that GPU until the process ends.  Host code never passes the
// array's name to a kernel (that is a host-side stand-in): it uses the
// device address hipGetSymbolAddress returns, looked up once per device.
__device__ __align__(256) unsigned char scratch[TAURUS_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

void* scratch_of_current_device() {
    int dev = 0;
    TAURUS_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= MAX_DEVICES) fail(TAURUS_E_DEVICE, "device %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t rc = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (rc != hipSuccess || !p)
            fail(TAURUS_E_DEVICE, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(rc));
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}
}  // namespace

// Scratch bytes the build takes for e edges, an upper bound: two key arrays,
// the first-digit histogram, and per radix pass at most 1,024 buckets of
// 4-byte counts per tile, plus the offset computation's per-group counts and
// offsets (at most ceil(sqrt(tiles)) groups) and digit totals, each block
// rounded to 256 bytes.
int64_t build_csr_scratch_bytes(int64_t e) {
    const int64_t tiles = ceil_div(std::max<int64_t>(e, 1), RADIX_TILE);
    const int64_t buckets = 1024 * tiles;
    int64_t groups = 1;
    while (groups * groups < tiles) groups++;
    return 256 + 2 * (8 * std::max<int64_t>(e, 1) + 256) + (1024 * tiles + 256) + (4 * buckets + 256) +
           2 * (8 * 1024 * groups + 256) + (8 * 1024 + 256) + 4096;
}

int build_csr_noalloc_impl(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                           int32_t* col_dst, hipStream_t s) {
    check_build_args(n, e, src, dst, row_off, col_dst);
    if (e > TAURUS_NOALLOC_MAX_EDGES || build_csr_scratch_bytes(e) > TAURUS_NOALLOC_SCRATCH_BYTES)
        fail(TAURUS_E_INVALID, "taurus_build_csr_noalloc: %lld edges exceed the limit of %lld", (long long)e,
             (long long)TAURUS_NOALLOC_MAX_EDGES);
    void* base = scratch_of_current_device();
    Arena arena(s, base, TAURUS_NOALLOC_SCRATCH_BYTES);
    int* bad = enqueue_build_csr(arena, n, e, src, dst, row_off, col_dst, s);
    int hbad = 0;
    TAURUS_HIP(hipMemcpyAsync(&hbad, bad, sizeof(int), hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    report_build_flags(hbad);
    return TAURUS_OK;
}

}  // namespace taurus
