// Device-wide primitives used while building graph structures: an exclusive
// prefix sum and a stable LSD radix sort of 64-bit keys with 32-bit values.
// Both are written for wave64: wave-level scans use cross-lane shuffles and
// the radix ranking matches digits within a wave with eight ballots.
#include <algorithm>
#include <chrono>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <mutex>
#include <unordered_map>

#include "internal.hpp"

namespace taurus {

// ---------------------------------------------------------------- errors ----
static thread_local std::string g_last_error;

void set_error(const char* fmt, ...) {
    char buf[1024];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
}

void fail(int status, const char* fmt, ...) {
    char buf[1024];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    throw Failure{status};
}

const char* last_error_cstr() { return g_last_error.c_str(); }

// ------------------------------------------------------ device memory cache --
// Device memory comes from hipMalloc once and is then recycled.  A released
// block goes to a free list keyed by (device, size class) with the stream it
// was released on and an event recorded there.  A later request of the same
// class takes it at once on that stream (stream order covers the earlier
// use), or on another stream after making that stream wait for the event.
// Requests are rounded up to a class (at most 1/8 above the request), so
// buffers of similar size share blocks.  On hipMalloc failure every cached
// block of the device is returned to the driver and the request retried once.
namespace {

struct FreeBlock {
    void* p;
    hipStream_t s;
};

struct BlockInfo {
    int dev;
    size_t cls;
    hipEvent_t ev;  // recorded on release; created on the first release
};

struct DeviceCache {
    std::mutex mu;
    std::map<std::pair<int, size_t>, std::vector<FreeBlock>> free_lists;
    std::unordered_map<void*, BlockInfo> blocks;  // every block obtained from hipMalloc
};

// lives until the process ends: blocks may be released from static destructors
DeviceCache& device_cache() {
    static DeviceCache* c = new DeviceCache();
    return *c;
}

size_t size_class(size_t bytes) {
    if (bytes <= 4096) return 4096;
    const int k = 63 - __builtin_clzll((unsigned long long)bytes);  // 2^k <= bytes
    const size_t step = (size_t)1 << std::max(k - 3, 12);
    return (bytes + step - 1) / step * step;
}

// TAURUS_ALLOC_LOG=1: one line on stderr per hipMalloc, hipFree and trim
// of the device memory cache, with its size and wall time
bool alloc_log() {
    static const bool on = [] {
        const char* v = std::getenv("TAURUS_ALLOC_LOG");
        return v && v[0] == '1';
    }();
    return on;
}

double ms_now() {
    return std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now().time_since_epoch()).count();
}

// hipFree cached blocks of device dev, smallest first, until at least
// `need` bytes are freed or none is left; returns the bytes freed.  Large
// blocks are kept when small ones suffice: re-allocating a freed block of
// tens of GB costs seconds.  The caller holds no lock.
size_t trim_device(int dev, size_t need) {
    DeviceCache& c = device_cache();
    const double t0 = alloc_log() ? ms_now() : 0.0;
    size_t freed = 0;
    (void)hipDeviceSynchronize();
    std::lock_guard<std::mutex> g(c.mu);
    // free_lists is ordered by (device, size class)
    for (auto it = c.free_lists.lower_bound({dev, 0});
         it != c.free_lists.end() && it->first.first == dev && freed < need;) {
        std::vector<FreeBlock>& v = it->second;
        while (!v.empty() && freed < need) {
            const FreeBlock b = v.back();
            v.pop_back();
            auto bi = c.blocks.find(b.p);
            if (bi != c.blocks.end()) {
                if (bi->second.ev) (void)hipEventDestroy(bi->second.ev);
                c.blocks.erase(bi);
            }
            (void)hipFree(b.p);
            freed += it->first.second;
        }
        if (v.empty()) it = c.free_lists.erase(it);
        else ++it;
    }
    (void)hipGetLastError();
    if (alloc_log()) std::fprintf(stderr, "[taurus alloc] trim: %.3f GB freed in %.1f ms\n", freed / 1e9, ms_now() - t0);
    return freed;
}

}  // namespace

// requests of at least this size may reuse a larger cached block
constexpr size_t OVERSIZE_MIN = (size_t)64 << 20;

void* device_acquire(size_t bytes, hipStream_t s, size_t* got, bool may_oversize) {
    int dev = 0;
    TAURUS_HIP(hipGetDevice(&dev));
    const size_t cls = size_class(bytes);
    *got = cls;
    DeviceCache& c = device_cache();
    {
        std::lock_guard<std::mutex> g(c.mu);
        auto it = c.free_lists.find({dev, cls});
        if ((it == c.free_lists.end() || it->second.empty()) && may_oversize && cls >= OVERSIZE_MIN) {
            // a large request may take the smallest cached block up to 1.5x
            // its class instead of a fresh hipMalloc
            for (auto j = c.free_lists.upper_bound({dev, cls});
                 j != c.free_lists.end() && j->first.first == dev && j->first.second <= cls + cls / 2; ++j)
                if (!j->second.empty()) {
                    it = j;
                    *got = j->first.second;
                    break;
                }
        }
        if (it != c.free_lists.end() && !it->second.empty()) {
            std::vector<FreeBlock>& v = it->second;
            size_t pick = v.size() - 1;
            for (size_t i = v.size(); i-- > 0;)
                if (v[i].s == s) {
                    pick = i;
                    break;
                }
            const FreeBlock b = v[pick];
            v.erase(v.begin() + (long)pick);
            if (b.s != s) TAURUS_HIP(hipStreamWaitEvent(s, c.blocks.at(b.p).ev, 0));
            return b.p;
        }
    }
    void* p = nullptr;
    const double t0 = alloc_log() ? ms_now() : 0.0;
    hipError_t e = hipMalloc(&p, cls);
    while (e == hipErrorOutOfMemory) {
        (void)hipGetLastError();
        if (alloc_log()) std::fprintf(stderr, "[taurus alloc] hipMalloc(%.3f GB) out of memory\n", cls / 1e9);
        if (trim_device(dev, cls) == 0) break;
        e = hipMalloc(&p, cls);
    }
    if (alloc_log())
        std::fprintf(stderr, "[taurus alloc] hipMalloc(%.3f GB): %s in %.1f ms\n", cls / 1e9,
                     e == hipSuccess ? "ok" : "failed", ms_now() - t0);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        fail(e == hipErrorOutOfMemory ? TAURUS_E_OOM : TAURUS_E_DEVICE, "hipMalloc(%zu) failed: %s", cls,
             hipGetErrorString(e));
    }
    std::lock_guard<std::mutex> g(c.mu);
    c.blocks[p] = BlockInfo{dev, cls, nullptr};
    return p;
}

size_t release_cached(size_t bytes) {
    int dev = 0;
    TAURUS_HIP(hipGetDevice(&dev));
    return trim_device(dev, bytes == 0 ? SIZE_MAX : bytes);
}

void device_release(void* p, hipStream_t s) {
    if (!p) return;
    DeviceCache& c = device_cache();
    std::lock_guard<std::mutex> g(c.mu);
    auto bi = c.blocks.find(p);
    if (bi == c.blocks.end()) return;
    BlockInfo& info = bi->second;
    if (!info.ev && hipEventCreateWithFlags(&info.ev, hipEventDisableTiming) != hipSuccess) {
        // no event: wait here so that any stream may take the block
        (void)hipGetLastError();
        info.ev = nullptr;
        (void)hipStreamSynchronize(s);
        (void)hipFree(p);
        c.blocks.erase(bi);
        return;
    }
    (void)hipEventRecord(info.ev, s);
    c.free_lists[{info.dev, info.cls}].push_back(FreeBlock{p, s});
}

// ---------------------------------------------------------- pinned blocks --
// Large pinned host buffers (the residency store for evicted rows, the chunk
// loader's ring) come from a cache as device memory does: pinning tens of
// GB costs seconds, and the next layer usually needs the same size.  A
// request takes the smallest free block at least as large.
namespace {
struct PinnedCache {
    std::mutex mu;
    std::multimap<size_t, void*> free;
};
PinnedCache& pinned_cache() {
    static PinnedCache* c = new PinnedCache;  // outlives every static destructor
    return *c;
}
}  // namespace

void* pinned_acquire(size_t bytes, size_t* cap) {
    bytes = std::max<size_t>(bytes, 1);
    {
        PinnedCache& c = pinned_cache();
        std::lock_guard<std::mutex> g(c.mu);
        auto it = c.free.lower_bound(bytes);
        if (it != c.free.end()) {
            void* p = it->second;
            *cap = it->first;
            c.free.erase(it);
            return p;
        }
    }
    void* p = nullptr;
    const hipError_t e = hipHostMalloc(&p, bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        fail(TAURUS_E_OOM, "pinned host allocation of %zu bytes failed: %s", bytes, hipGetErrorString(e));
    }
    *cap = bytes;
    return p;
}

void pinned_return(void* p, size_t cap) {
    if (!p) return;
    PinnedCache& c = pinned_cache();
    std::lock_guard<std::mutex> g(c.mu);
    c.free.emplace(cap, p);
}

size_t release_pinned() {
    PinnedCache& c = pinned_cache();
    std::lock_guard<std::mutex> g(c.mu);
    size_t total = 0;
    for (auto& kv : c.free) {
        (void)hipHostFree(kv.second);
        total += kv.first;
    }
    c.free.clear();
    return total;
}

// ------------------------------------------------------------ pinned staging --
// One pinned host buffer per host thread for small transfers, grown on demand
// and kept until the process ends.  An asynchronous transfer still reading
// it is tracked by one event.
namespace {
struct Staging {
    void* buf = nullptr;
    size_t cap = 0;
    hipEvent_t busy = nullptr;
    bool in_flight = false;
};
thread_local Staging t_stage;
}  // namespace

void* pinned_staging(size_t bytes) {
    Staging& st = t_stage;
    if (st.in_flight) {
        TAURUS_HIP(hipEventSynchronize(st.busy));
        st.in_flight = false;
    }
    if (bytes > st.cap) {
        size_t want = std::max<size_t>(bytes, 64 << 10);
        void* p = nullptr;
        TAURUS_HIP(hipHostMalloc(&p, want, hipHostMallocDefault));
        if (st.buf) (void)hipHostFree(st.buf);
        st.buf = p;
        st.cap = want;
    }
    return st.buf;
}

void pinned_staging_in_flight(hipStream_t s) {
    Staging& st = t_stage;
    if (!st.busy) TAURUS_HIP(hipEventCreateWithFlags(&st.busy, hipEventDisableTiming));
    TAURUS_HIP(hipEventRecord(st.busy, s));
    st.in_flight = true;
}

void Readback::add_bytes(void* host, const void* dev, size_t bytes) {
    items_.push_back({host, dev, bytes, total_});
    total_ += (bytes + 15) & ~(size_t)15;
}

void Readback::run(hipStream_t s) {
    if (items_.empty()) return;
    char* stage = static_cast<char*>(pinned_staging(total_));
    for (const Item& it : items_)
        TAURUS_HIP(hipMemcpyAsync(stage + it.off, it.dev, it.bytes, hipMemcpyDeviceToHost, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    for (const Item& it : items_) std::memcpy(it.host, stage + it.off, it.bytes);
    items_.clear();
    total_ = 0;
}

// ---------------------------------------------------------------- arena -----
void* Arena::alloc_bytes(int64_t bytes, const char* what) {
    if (bytes <= 0) bytes = 16;
    if (region_) {
        const int64_t start = (top_ + 255) & ~(int64_t)255;
        if (start + bytes <= capacity_ && nstarts_ < REGION_STACK) {
            starts_[nstarts_++] = top_;
            top_ = start + bytes;
            if (top_ > peak_) peak_ = top_;
            return region_ + start;
        }
        if (!fallback_)
            fail(TAURUS_E_INVALID, "scratch region of %lld bytes cannot hold %lld more bytes for %s",
                 (long long)capacity_, (long long)bytes, what);
    }
    const int64_t cls = (int64_t)size_class((size_t)bytes);
    if (budget_ > 0 && bytes_ + cls > budget_)
        fail(TAURUS_E_BUDGET, "allocating %lld bytes for %s exceeds the budget (%lld of %lld in use)",
             (long long)cls, what, (long long)bytes_, (long long)budget_);
    size_t got = 0;
    void* p = nullptr;
    try {
        p = device_acquire((size_t)bytes, stream_, &got, budget_ <= 0);
    } catch (const Failure&) {
        set_error("%s (for %s)", last_error_cstr(), what);
        throw;
    }
    // a block taken oversize is counted at the requested class
    got = std::min(got, (size_t)cls);
    blocks_.push_back({p, (int64_t)got});
    bytes_ += (int64_t)got;
    if (bytes_ > peak_) peak_ = bytes_;
    return p;
}

void Arena::free_ptr(void* p) {
    if (region_ && static_cast<char*>(p) >= region_ && static_cast<char*>(p) < region_ + capacity_) {
        // the most recent block only: its start was recorded before alignment
        if (nstarts_ > 0 && p == region_ + ((starts_[nstarts_ - 1] + 255) & ~(int64_t)255)) top_ = starts_[--nstarts_];
        return;
    }
    for (size_t i = blocks_.size(); i-- > 0;) {
        if (blocks_[i].p == p) {
            device_release(p, stream_);
            bytes_ -= blocks_[i].bytes;
            blocks_.erase(blocks_.begin() + (long)i);
            return;
        }
    }
}

void Arena::release() {
    if (region_) {
        top_ = 0;
        nstarts_ = 0;
    }
    for (auto& b : blocks_) device_release(b.p, stream_);
    blocks_.clear();
    bytes_ = 0;
}

// ----------------------------------------------------------------- fills ----
template <typename T>
__global__ void k_fill(T* __restrict__ p, int64_t n, T v) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

void fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
    if (n <= 0) return;
    k_fill<int32_t><<<(unsigned)ceil_div(n, 256), 256, 0, s>>>(p, n, v);
    TAURUS_CHECK_LAUNCH();
}

// ---------------------------------------------------------------- scan ------
constexpr int SCAN_THREADS = 256;
constexpr int SCAN_ITEMS = 16;
constexpr int SCAN_TILE = SCAN_THREADS * SCAN_ITEMS;

// inclusive scan across a wave64 with shuffles
__device__ inline uint64_t wave_incl_scan(uint64_t x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        uint64_t y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    return x;
}

// exclusive scan of one value per thread across the block; returns the
// block total in *total
__device__ inline uint64_t block_excl_scan(uint64_t x, uint64_t* total) {
    __shared__ uint64_t wsum[SCAN_THREADS / 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint64_t inc = wave_incl_scan(x);
    if (lane == 63) wsum[wave] = inc;
    __syncthreads();
    uint64_t before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < SCAN_THREADS / 64; w++) {
        if (w < wave) before += wsum[w];
        all += wsum[w];
    }
    __syncthreads();
    *total = all;
    return before + inc - x;
}

template <typename Tin>
__global__ __launch_bounds__(SCAN_THREADS) void k_scan_tile_sums(const Tin* __restrict__ in, int64_t n,
                                                                 uint64_t* __restrict__ sums) {
    const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
    uint64_t s = 0;
    for (int i = threadIdx.x; i < SCAN_TILE; i += SCAN_THREADS) {
        int64_t g = base + i;
        if (g < n) s += (uint64_t)in[g];
    }
    uint64_t total;
    (void)block_excl_scan(s, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

template <typename Tin, typename Tout>
__global__ __launch_bounds__(SCAN_THREADS) void k_scan_tile_apply(const Tin* __restrict__ in, int64_t n,
                                                                  const uint64_t* __restrict__ offsets,
                                                                  Tout* __restrict__ out) {
    __shared__ uint64_t stage[SCAN_TILE];
    const int64_t base = (int64_t)blockIdx.x * SCAN_TILE;
    for (int i = threadIdx.x; i < SCAN_TILE; i += SCAN_THREADS) {
        int64_t g = base + i;
        stage[i] = g < n ? (uint64_t)in[g] : 0;
    }
    __syncthreads();
    uint64_t v[SCAN_ITEMS];
    uint64_t s = 0;
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; j++) {
        v[j] = stage[threadIdx.x * SCAN_ITEMS + j];
        s += v[j];
    }
    uint64_t total;
    uint64_t run = block_excl_scan(s, &total) + (offsets ? offsets[blockIdx.x] : 0);
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; j++) {
        stage[threadIdx.x * SCAN_ITEMS + j] = run;
        run += v[j];
    }
    __syncthreads();
    for (int i = threadIdx.x; i < SCAN_TILE; i += SCAN_THREADS) {
        int64_t g = base + i;
        if (g < n) out[g] = (Tout)stage[i];
    }
}

// Exclusive scan of a short sequence (the tile sums) by one workgroup that
// walks it a tile at a time with a running carry: one launch instead of
// another level of tiles.
__global__ __launch_bounds__(SCAN_THREADS) void k_scan_serial(const uint64_t* __restrict__ in, int64_t n,
                                                              uint64_t* __restrict__ out) {
    __shared__ uint64_t stage[SCAN_TILE];
    uint64_t carry = 0;
    for (int64_t base = 0; base < n; base += SCAN_TILE) {
        for (int i = threadIdx.x; i < SCAN_TILE; i += SCAN_THREADS) stage[i] = base + i < n ? in[base + i] : 0;
        __syncthreads();
        uint64_t v[SCAN_ITEMS];
        uint64_t s = 0;
#pragma unroll
        for (int j = 0; j < SCAN_ITEMS; j++) {
            v[j] = stage[threadIdx.x * SCAN_ITEMS + j];
            s += v[j];
        }
        uint64_t total;
        uint64_t run = block_excl_scan(s, &total) + carry;
#pragma unroll
        for (int j = 0; j < SCAN_ITEMS; j++) {
            stage[threadIdx.x * SCAN_ITEMS + j] = run;
            run += v[j];
        }
        __syncthreads();
        for (int i = threadIdx.x; i < SCAN_TILE; i += SCAN_THREADS)
            if (base + i < n) out[base + i] = stage[i];
        __syncthreads();  // stage is reloaded for the next tile
        carry += total;
    }
}
constexpr int64_t SCAN_SERIAL_MAX = 1 << 16;  // tile sums scanned by k_scan_serial

template <typename Tout>
__global__ void k_write_total(const uint64_t* __restrict__ sums_scanned, const uint64_t* __restrict__ sums,
                              int64_t nb, Tout* __restrict__ out, int64_t n) {
    if (threadIdx.x == 0 && blockIdx.x == 0) out[n] = (Tout)(sums_scanned[nb - 1] + sums[nb - 1]);
}
template <typename Tout>
__global__ void k_write_zero(Tout* __restrict__ out) {
    if (threadIdx.x == 0 && blockIdx.x == 0) out[0] = 0;
}

// exclusive scan of n values (any integer type) into out (uint64/int64)
template <typename Tin, typename Tout>
static void scan_impl(const Tin* in, Tout* out, int64_t n, bool write_total, Arena& arena, hipStream_t s) {
    if (n == 0) {
        if (write_total) {
            k_write_zero<<<1, 64, 0, s>>>(out);
            TAURUS_CHECK_LAUNCH();
        }
        return;
    }
    const int64_t nb = ceil_div(n, SCAN_TILE);
    uint64_t* sums = arena.alloc<uint64_t>(nb, "scan block sums");
    uint64_t* sums_scanned = arena.alloc<uint64_t>(nb, "scan block offsets");
    k_scan_tile_sums<Tin><<<(unsigned)nb, SCAN_THREADS, 0, s>>>(in, n, sums);
    TAURUS_CHECK_LAUNCH();
    if (nb <= SCAN_SERIAL_MAX) {
        k_scan_serial<<<1, SCAN_THREADS, 0, s>>>(sums, nb, sums_scanned);
        TAURUS_CHECK_LAUNCH();
    } else {
        scan_impl<uint64_t, uint64_t>(sums, sums_scanned, nb, false, arena, s);
    }
    k_scan_tile_apply<Tin, Tout><<<(unsigned)nb, SCAN_THREADS, 0, s>>>(in, n, sums_scanned, out);
    TAURUS_CHECK_LAUNCH();
    if (write_total) {
        k_write_total<Tout><<<1, 64, 0, s>>>(sums_scanned, sums, nb, out, n);
        TAURUS_CHECK_LAUNCH();
    }
    arena.free_ptr(sums_scanned);
    arena.free_ptr(sums);
}

void scan_u32_to_u64(const uint32_t* in, uint64_t* out, int64_t n, bool write_total, Arena& arena,
                     hipStream_t s) {
    scan_impl<uint32_t, uint64_t>(in, out, n, write_total, arena, s);
}
void scan_i32_to_i64(const int32_t* in, int64_t* out, int64_t n, bool write_total, Arena& arena,
                     hipStream_t s) {
    scan_impl<int32_t, int64_t>(in, out, n, write_total, arena, s);
}
void scan_u64(const uint64_t* in, uint64_t* out, int64_t n, bool write_total, Arena& arena, hipStream_t s) {
    scan_impl<uint64_t, uint64_t>(in, out, n, write_total, arena, s);
}

// ---------------------------------------------------------------- radix -----
constexpr int RS_THREADS = 256;
constexpr int RS_ITEMS = 16;
constexpr int RS_TILE = RS_THREADS * RS_ITEMS;
constexpr int RS_WAVES = RS_THREADS / 64;

// Digits are DBITS wide (8, 9 or 10): NB = 2^DBITS buckets, each of the
// block's 256 threads owning Q = NB / 256 consecutive buckets wherever the
// kernels walk buckets.

// Lanes of a wave holding the same digit d: one ballot per digit bit.
template <int DBITS>
__device__ inline uint64_t digit_peers(uint32_t d, bool valid) {
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int bt = 0; bt < DBITS; bt++) {
        const bool bit = (d >> bt) & 1u;
        const uint64_t m = __ballot(bit);
        peers &= bit ? m : ~m;
    }
    return peers;
}

// Per tile: count of each digit (LDS atomics; the tile's loads are issued
// before any of them).  hist[tile * NB + b]: a tile's counts are one
// contiguous row, written and later read whole (a digit-major layout puts
// each count of a tile on its own cache line).
template <int DBITS, class K>
__global__ __launch_bounds__(RS_THREADS) void k_radix_hist(const K* __restrict__ keys, int64_t n,
                                                           int shift, int64_t nblocks,
                                                           uint32_t* __restrict__ hist) {
    constexpr int NB = 1 << DBITS, Q = NB / RS_THREADS;
    constexpr uint32_t MASK = NB - 1;
    __shared__ uint32_t h[NB];
#pragma unroll
    for (int q = 0; q < Q; q++) h[q * RS_THREADS + threadIdx.x] = 0;
    const int64_t base = (int64_t)blockIdx.x * RS_TILE;
    uint32_t d[RS_ITEMS];
#pragma unroll
    for (int r = 0; r < RS_ITEMS; r++) {
        const int64_t g = base + r * RS_THREADS + threadIdx.x;
        d[r] = g < n ? (uint32_t)((keys[g] >> shift) & MASK) : (uint32_t)NB;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < RS_ITEMS; r++)
        if (d[r] < (uint32_t)NB) atomicAdd(&h[d[r]], 1u);
    __syncthreads();
#pragma unroll
    for (int q = 0; q < Q; q++) {
        const int bkt = q * RS_THREADS + threadIdx.x;
        hist[(int64_t)blockIdx.x * NB + bkt] = h[bkt];
    }
}

// The global position of a tile's first item of digit d is (items of
// digits < d) + (items of digit d in tiles before this one).  From the
// tile-major histogram, over groups of `gt` consecutive tiles, it is kept as
// a group base gb[group * NB + d] (64-bit) plus the tile's offset within its
// group, written over the tile's count (32-bit: a group holds fewer than
// 2^32 items), in three steps:
//   k_radix_group_sums: per group, each digit's count;
//   k_radix_digit_scan: per digit, the exclusive prefix of those counts over
//     the groups, and the digit's total (a workgroup per 64 digits, its four
//     waves taking a quarter of the groups each);
//   k_radix_offsets: per group, the digits' bases (an exclusive scan of the
//     totals) plus the group's prefix into gb, then the group's tiles one
//     after another, each count replaced by the running offset.
template <int DBITS>
__global__ __launch_bounds__(RS_THREADS) void k_radix_group_sums(const uint32_t* __restrict__ hist, int64_t nblocks,
                                                                 int64_t gt, uint64_t* __restrict__ gsum) {
    constexpr int NB = 1 << DBITS, Q = NB / RS_THREADS;
    const int64_t t0 = (int64_t)blockIdx.x * gt, t1 = min(t0 + gt, nblocks);
    uint64_t acc[Q] = {};
    int64_t t = t0;
    for (; t + 4 <= t1; t += 4) {  // four rows' loads in flight
        uint32_t x[4][Q];
#pragma unroll
        for (int u = 0; u < 4; u++)
#pragma unroll
            for (int q = 0; q < Q; q++) x[u][q] = hist[(t + u) * NB + q * RS_THREADS + threadIdx.x];
#pragma unroll
        for (int u = 0; u < 4; u++)
#pragma unroll
            for (int q = 0; q < Q; q++) acc[q] += x[u][q];
    }
    for (; t < t1; t++)
#pragma unroll
        for (int q = 0; q < Q; q++) acc[q] += hist[t * NB + q * RS_THREADS + threadIdx.x];
#pragma unroll
    for (int q = 0; q < Q; q++) gsum[(int64_t)blockIdx.x * NB + q * RS_THREADS + threadIdx.x] = acc[q];
}

template <int DBITS>
__global__ __launch_bounds__(RS_THREADS) void k_radix_digit_scan(const uint64_t* __restrict__ gsum, int64_t ng,
                                                                 uint64_t* __restrict__ gscan,
                                                                 uint64_t* __restrict__ tot) {
    constexpr int NB = 1 << DBITS;
    __shared__ uint64_t wpart[RS_WAVES][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int d = blockIdx.x * 64 + lane;  // NB is a multiple of 64
    const int64_t per = (ng + RS_WAVES - 1) / RS_WAVES;
    const int64_t g0 = min((int64_t)wave * per, ng), g1 = min(g0 + per, ng);
    uint64_t sum = 0;
    for (int64_t g = g0; g < g1; g++) sum += gsum[g * NB + d];
    wpart[wave][lane] = sum;
    __syncthreads();
    uint64_t run = 0, all = 0;
#pragma unroll
    for (int w = 0; w < RS_WAVES; w++) {
        if (w < wave) run += wpart[w][lane];
        all += wpart[w][lane];
    }
    for (int64_t g = g0; g < g1; g++) {
        gscan[g * NB + d] = run;
        run += gsum[g * NB + d];
    }
    if (wave == 0) tot[d] = all;
}

template <int DBITS>
__global__ __launch_bounds__(RS_THREADS) void k_radix_offsets(uint32_t* __restrict__ hist, int64_t nblocks,
                                                              int64_t gt, const uint64_t* __restrict__ gscan,
                                                              const uint64_t* __restrict__ tot,
                                                              uint64_t* __restrict__ gb) {
    constexpr int NB = 1 << DBITS, Q = NB / RS_THREADS;
    __shared__ uint64_t wsum[RS_WAVES];
    __shared__ uint64_t base[NB];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // digit bases: thread t owns digits [t*Q, t*Q + Q)
    uint64_t own = 0, tq[Q];
#pragma unroll
    for (int q = 0; q < Q; q++) {
        tq[q] = tot[tid * Q + q];
        own += tq[q];
    }
    uint64_t incl = own;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint64_t y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    uint64_t b = incl - own;
#pragma unroll
    for (int w = 0; w < RS_WAVES; w++)
        if (w < wave) b += wsum[w];
#pragma unroll
    for (int q = 0; q < Q; q++) {
        base[tid * Q + q] = b;
        b += tq[q];
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < Q; q++) {
        const int64_t i = (int64_t)blockIdx.x * NB + q * RS_THREADS + tid;
        gb[i] = base[q * RS_THREADS + tid] + gscan[i];
    }
    const int64_t t0 = (int64_t)blockIdx.x * gt, t1 = min(t0 + gt, nblocks);
    uint32_t run[Q] = {};
    int64_t t = t0;
    for (; t + 4 <= t1; t += 4) {  // four rows' loads in flight
        uint32_t x[4][Q];
#pragma unroll
        for (int u = 0; u < 4; u++)
#pragma unroll
            for (int q = 0; q < Q; q++) x[u][q] = hist[(t + u) * NB + q * RS_THREADS + tid];
#pragma unroll
        for (int u = 0; u < 4; u++)
#pragma unroll
            for (int q = 0; q < Q; q++) {
                hist[(t + u) * NB + q * RS_THREADS + tid] = run[q];
                run[q] += x[u][q];
            }
    }
    for (; t < t1; t++)
#pragma unroll
        for (int q = 0; q < Q; q++) {
            const int64_t i = t * NB + q * RS_THREADS + tid;
            const uint32_t x = hist[i];
            hist[i] = run[q];
            run[q] += x;
        }
}

// tiles per group of the offset computation: about the square root of the
// tile count, so that the per-digit scan over groups and each group's walk
// over its tiles are about equally long
static int64_t radix_group_tiles(int64_t nblocks) {
    int64_t g = 1;
    while (g * g < nblocks) g++;
    return g;
}

// Scatter one tile stably, staged through LDS so that each digit's items
// leave the block as one contiguous run.  Wave w ranks the tile's items
// [w * RS_WITEMS, (w + 1) * RS_WITEMS) in index order, 64 per round: a lane's
// rank is the wave's running count of its digit plus its rank among the
// lanes holding that digit (digit match).  The waves' counts are then scanned
// per digit, so wave w's items of digit d follow those of waves < w, and the
// digit's start within the tile comes from the tile histogram.  The ranked
// tile is written to LDS in digit order and copied out: LDS slot i of digit
// d goes to offs[d] + (i - start of d in the tile).  Values take a second
// trip through the same LDS array after the keys (one array keeps the
// block's LDS at about 40 KB, four blocks per CU); each thread remembers the
// digits of the slots it copied out.
constexpr int RS_WITEMS = RS_TILE / RS_WAVES;   // items per wave
constexpr int RS_COPY = RS_TILE / RS_THREADS;   // slots each thread copies out
template <int DBITS, class K>
__global__ __launch_bounds__(RS_THREADS) void k_radix_scatter(
    const K* __restrict__ kin, const uint32_t* __restrict__ vin, int64_t n, int shift,
    const uint32_t* __restrict__ rel, const uint64_t* __restrict__ gb, int64_t gt,
    K* __restrict__ kout, uint32_t* __restrict__ vout, int* __restrict__ bad, int bad_bit) {
    constexpr int NB = 1 << DBITS, Q = NB / RS_THREADS;
    constexpr uint32_t MASK = NB - 1;
    __shared__ K skey[RS_TILE];
    __shared__ uint64_t gbase[NB];
    __shared__ uint32_t dstart[NB];
    __shared__ uint32_t wcnt[RS_WAVES][NB];   // per wave: running count, then its offset within the digit
    __shared__ uint32_t wsum[RS_WAVES];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t tile0 = (int64_t)blockIdx.x * RS_TILE;
    const int count = (int)min((int64_t)RS_TILE, n - tile0);
    const int wbase = wave * RS_WITEMS;

    // the tile's global offsets (its group's base plus its offset within
    // the group; thread t owning buckets [t*Q, t*Q + Q)) are requested first
    uint64_t go[Q];
#pragma unroll
    for (int q = 0; q < Q; q++) {
        const int d = tid * Q + q;
        go[q] = gb[(int64_t)(blockIdx.x / gt) * NB + d] + rel[(int64_t)blockIdx.x * NB + d];
    }
    K keys[RS_ITEMS];
    uint32_t vals[RS_ITEMS];
#pragma unroll
    for (int r = 0; r < RS_ITEMS; r++) {
        const int li = wbase + r * 64 + lane;
        keys[r] = li < count ? kin[tile0 + li] : 0;
        vals[r] = (li < count && vin) ? vin[tile0 + li] : 0;
    }
#pragma unroll
    for (int w = 0; w < RS_WAVES; w++)
#pragma unroll
        for (int q = 0; q < Q; q++) wcnt[w][q * RS_THREADS + tid] = 0;
#pragma unroll
    for (int q = 0; q < Q; q++) gbase[tid * Q + q] = go[q];
    __syncthreads();

    // rank within the wave (no block barrier: the counters are the wave's own)
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    uint32_t rank[RS_ITEMS];
#pragma unroll
    for (int r = 0; r < RS_ITEMS; r++) {
        const bool valid = wbase + r * 64 + lane < count;
        const uint32_t d = (uint32_t)((keys[r] >> shift) & MASK);
        const uint64_t peers = digit_peers<DBITS>(d, valid);
        const uint32_t runc = valid ? wcnt[wave][d] : 0u;
        rank[r] = runc + (uint32_t)__popcll(peers & lt_mask);
        if (valid && (peers & lt_mask) == 0) wcnt[wave][d] = runc + (uint32_t)__popcll(peers);
    }
    __syncthreads();
    // the tile's count of each digit is the sum of the waves' counts; the
    // digits' starts within the tile are their exclusive scan
    uint32_t hq[Q], own = 0;
#pragma unroll
    for (int q = 0; q < Q; q++) {
        hq[q] = 0;
#pragma unroll
        for (int w = 0; w < RS_WAVES; w++) hq[q] += wcnt[w][tid * Q + q];
        own += hq[q];
    }
    uint32_t incl = own;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(incl, off, 64);
        if (lane >= off) incl += y;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    uint32_t run = incl - own;
#pragma unroll
    for (int w = 0; w < RS_WAVES; w++)
        if (w < wave) run += wsum[w];
    // per digit: the start of the digit in the tile and the waves' offsets
    // within its run (thread t's own digits: no other thread reads them here)
#pragma unroll
    for (int q = 0; q < Q; q++) {
        const int bkt = tid * Q + q;
        dstart[bkt] = run;
        uint32_t acc = run;
#pragma unroll
        for (int w = 0; w < RS_WAVES; w++) {
            const uint32_t c = wcnt[w][bkt];
            wcnt[w][bkt] = acc;
            acc += c;
        }
        run += hq[q];
    }
    __syncthreads();
    // LDS slot of each item (count or more: out of range, flagged)
#pragma unroll
    for (int r = 0; r < RS_ITEMS; r++) {
        if (wbase + r * 64 + lane >= count) {
            rank[r] = RS_TILE;
            continue;
        }
        const uint32_t d = (uint32_t)((keys[r] >> shift) & MASK);
        rank[r] = wcnt[wave][d] + rank[r];
        if (rank[r] < (uint32_t)count) skey[rank[r]] = keys[r];
        else atomicOr(bad, bad_bit);
    }
    __syncthreads();
    uint32_t dig[RS_COPY];
#pragma unroll
    for (int j = 0; j < RS_COPY; j++) {
        const int i = j * RS_THREADS + tid;
        dig[j] = 0;
        if (i < count) {
            const K key = skey[i];
            const uint32_t d = (uint32_t)((key >> shift) & MASK);
            dig[j] = d;
            const uint64_t pos = gbase[d] + (uint64_t)(i - (int)dstart[d]);
            if (pos < (uint64_t)n) kout[pos] = key;
            else atomicOr(bad, bad_bit);
        }
    }
    if (!vin) return;
    __syncthreads();  // every key is out of LDS
    uint32_t* sval = reinterpret_cast<uint32_t*>(skey);
#pragma unroll
    for (int r = 0; r < RS_ITEMS; r++)
        if (rank[r] < (uint32_t)count) sval[rank[r]] = vals[r];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < RS_COPY; j++) {
        const int i = j * RS_THREADS + tid;
        if (i < count) {
            const uint32_t d = dig[j];
            const uint64_t pos = gbase[d] + (uint64_t)(i - (int)dstart[d]);
            if (pos < (uint64_t)n) vout[pos] = sval[i];
        }
    }
}

template <int DBITS, class K>
static void radix_pass(SortBuffersT<K>& b, int64_t n, int shift, int64_t nblocks, uint32_t* pre, uint32_t* hist,
                       Arena& arena, hipStream_t s, int* bad, int bad_bit) {
    constexpr int NB = 1 << DBITS;
    const int c = b.cur;
    if (pre) {  // the tile histogram of this digit came with the keys
        hist = pre;
    } else {
        k_radix_hist<DBITS, K><<<(unsigned)nblocks, RS_THREADS, 0, s>>>(b.keys[c], n, shift, nblocks, hist);
        TAURUS_CHECK_LAUNCH();
    }
    const int64_t gt = radix_group_tiles(nblocks), ng = ceil_div(nblocks, gt);
    uint64_t* gsum = arena.alloc<uint64_t>(ng * NB, "radix group counts");
    uint64_t* gscan = arena.alloc<uint64_t>(ng * NB, "radix group offsets");
    uint64_t* tot = arena.alloc<uint64_t>(NB, "radix digit totals");
    k_radix_group_sums<DBITS><<<(unsigned)ng, RS_THREADS, 0, s>>>(hist, nblocks, gt, gsum);
    TAURUS_CHECK_LAUNCH();
    k_radix_digit_scan<DBITS><<<NB / 64, RS_THREADS, 0, s>>>(gsum, ng, gscan, tot);
    TAURUS_CHECK_LAUNCH();
    uint64_t* gb = gsum;  // the group counts are read once, by the digit scan
    k_radix_offsets<DBITS><<<(unsigned)ng, RS_THREADS, 0, s>>>(hist, nblocks, gt, gscan, tot, gb);
    TAURUS_CHECK_LAUNCH();
    k_radix_scatter<DBITS, K><<<(unsigned)nblocks, RS_THREADS, 0, s>>>(b.keys[c], b.vals[c], n, shift, hist, gb, gt,
                                                                       b.keys[1 - c], b.vals[1 - c], bad, bad_bit);
    TAURUS_CHECK_LAUNCH();
    arena.free_ptr(tot);
    arena.free_ptr(gscan);
    arena.free_ptr(gsum);
    b.cur = 1 - c;
}

// Digit schedule: 8-bit passes, the cheapest per sorted bit here (measured
// per pass at 20M key-value pairs with hist and scan: 8 bits ~190 us, 9 bits
// ~240 us; keys alone, 8 bits ~150 us); one pass fewer with some digits
// widened to 9 or 10 bits when that costs less, e.g. 25 bits as 9 + 8 + 8
// instead of four 8-bit passes.  Bits above key_bits are zero in every key sorted here, so a
// pass may cover a few more bits than remain.
static std::vector<int> digit_schedule(int key_bits) {
    const double cost[11] = {0, 0, 0, 0, 0, 0, 0, 0, 1.0, 1.27, 1.5};
    const int p8 = (key_bits + 7) / 8;
    std::vector<int> all8((size_t)p8, 8);
    const int p = p8 - 1;
    if (p < 1 || key_bits > 10 * p) return all8;
    std::vector<int> w((size_t)p, 8);
    for (int extra = key_bits - 8 * p, i = 0; extra > 0; i = (i + 1) % p, extra--) w[(size_t)i]++;
    double c = 0;
    for (int x : w) c += cost[x];
    return c < p8 * cost[8] ? w : all8;
}

static_assert(RS_TILE == RADIX_TILE, "producers of first_hist tile the keys like the sort");
template <class K>
static void radix_sort_impl(SortBuffersT<K>& b, int64_t n, int key_bits, Arena& arena, hipStream_t s, int* bad,
                            int bad_bit, uint32_t* first_hist, int first_bit) {
    if (n <= 1 || key_bits <= 0) return;
    const int64_t nblocks = ceil_div(n, RS_TILE);
    if (nblocks > 0x7fffffff) fail(TAURUS_E_INVALID, "radix sort of %lld items is too large", (long long)n);
    const std::vector<int> widths = digit_schedule(key_bits);
    const int wmax = *std::max_element(widths.begin(), widths.end());
    uint32_t* hist = arena.alloc<uint32_t>(((int64_t)1 << wmax) * nblocks, "radix histogram");
    int shift = first_bit;
    for (int width : widths) {
        if (shift >= (int)(8 * sizeof(K))) break;  // the remaining bits are zero in every key
        uint32_t* pre = shift == 0 && width == 8 ? first_hist : nullptr;
        if (width == 8) radix_pass<8, K>(b, n, shift, nblocks, pre, hist, arena, s, bad, bad_bit);
        else if (width == 9) radix_pass<9, K>(b, n, shift, nblocks, nullptr, hist, arena, s, bad, bad_bit);
        else radix_pass<10, K>(b, n, shift, nblocks, nullptr, hist, arena, s, bad, bad_bit);
        shift += width;
    }
    arena.free_ptr(hist);
}

void radix_sort_u64(SortBuffers& b, int64_t n, int key_bits, Arena& arena, hipStream_t s, int* bad,
                    int bad_bit, uint32_t* first_hist, int first_bit) {
    radix_sort_impl<uint64_t>(b, n, key_bits, arena, s, bad, bad_bit, first_hist, first_bit);
}

void radix_sort_u32(SortBuffers32& b, int64_t n, int key_bits, Arena& arena, hipStream_t s, int* bad, int bad_bit) {
    if (key_bits > 32) fail(TAURUS_E_INVALID, "32-bit radix sort of %d-bit keys", key_bits);
    radix_sort_impl<uint32_t>(b, n, key_bits, arena, s, bad, bad_bit, nullptr, 0);
}

}  // namespace taurus
