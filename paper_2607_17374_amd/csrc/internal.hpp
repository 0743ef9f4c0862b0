// Internal helpers of the HIP library: status propagation, error text,
// tracked device allocations and the primitive entry points shared by the
// translation units (scan, radix sort).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <chrono>
#include <cstring>
#include <memory>
#include <string>
#include <vector>

#include "../../include/taurus.h"

namespace taurus {

void set_error(const char* fmt, ...);

// Thrown inside the library only; every C entry point catches it.
struct Failure {
    int status;
};

[[noreturn]] void fail(int status, const char* fmt, ...);

#define TAURUS_HIP(expr)                                                                   \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess) {                                                            \
            ::taurus::fail(e_ == hipErrorOutOfMemory ? TAURUS_E_OOM : TAURUS_E_DEVICE,     \
                           "%s failed: %s (%s:%d)", #expr, hipGetErrorString(e_), __FILE__, \
                           __LINE__);                                                      \
        }                                                                                  \
    } while (0)

#define TAURUS_CHECK_LAUNCH() TAURUS_HIP(hipGetLastError())

// Device memory cache (prims.hip): device_acquire returns a block of at
// least `bytes` usable in stream order on `s` (*got = its size);
// device_release hands it back after the work queued on `s` so far.
// may_oversize: a request of 64 MB or more may take a cached block of up to
// 1.5 times its size class (*got then names the block's class).
void* device_acquire(size_t bytes, hipStream_t s, size_t* got, bool may_oversize = false);
void device_release(void* p, hipStream_t s);
// hipFree cached (unused) blocks of the current device, smallest first,
// until at least `bytes` are freed (0: all); returns the bytes freed
size_t release_cached(size_t bytes);

// Large pinned host buffers from a process-wide cache: a block of at least
// `bytes` (*cap receives its size), given back with pinned_return(p, cap)
// once nothing reads it; release_pinned frees every cached block.
void* pinned_acquire(size_t bytes, size_t* cap);
void pinned_return(void* p, size_t cap);
size_t release_pinned();

// Pinned host buffer of at least `bytes` for the calling thread (reused by
// its next call, which first waits for a transfer left in flight by
// pinned_staging_in_flight).
void* pinned_staging(size_t bytes);
// The thread's staging buffer is read by a transfer enqueued on s: the next
// pinned_staging call waits for it instead of the caller synchronising now.
void pinned_staging_in_flight(hipStream_t s);

// Small device-to-host reads gathered into one pinned transfer and one
// stream synchronisation: add() any number, then run().
class Readback {
public:
    // count elements of type T; host and device types must match (no
    // untyped overload, so a mismatch does not compile)
    template <typename T>
    void add(T* host, const T* dev, int64_t count) {
        add_bytes(static_cast<void*>(host), static_cast<const void*>(dev), (size_t)count * sizeof(T));
    }
    void run(hipStream_t s);

private:
    void add_bytes(void* host, const void* dev, size_t bytes);
    struct Item {
        void* host;
        const void* dev;
        size_t bytes, off;
    };
    std::vector<Item> items_;
    size_t total_ = 0;
};

// Device allocations owned by one object, with a byte budget, taken from and
// returned to the device memory cache on the owner's stream, so objects
// created one after another recycle each other's buffers.
class Arena {
public:
    explicit Arena(hipStream_t s = nullptr, int64_t budget = 0) : stream_(s), budget_(budget) {}
    // Fixed-region mode: allocations are carved, 256-byte aligned, out of
    // [region, region + capacity) and never touch the device memory cache;
    // running out is an error (TAURUS_E_INVALID), or, with fallback, a
    // request that does not fit comes from the cache as usual.  free_ptr
    // gives back the most recent block of the region only.
    Arena(hipStream_t s, void* region, int64_t capacity, bool fallback = false)
        : stream_(s), region_(static_cast<char*>(region)), capacity_(capacity), fallback_(fallback) {}
    ~Arena() { release(); }
    void set_stream(hipStream_t s) { stream_ = s; }
    Arena(const Arena&) = delete;
    Arena& operator=(const Arena&) = delete;

    template <typename T>
    T* alloc(int64_t count, const char* what) {
        return static_cast<T*>(alloc_bytes(count * (int64_t)sizeof(T), what));
    }
    void* alloc_bytes(int64_t bytes, const char* what);
    void free_ptr(void* p);
    void release();
    void set_budget(int64_t budget) { budget_ = budget; }
    int64_t bytes() const { return bytes_; }
    int64_t peak() const { return peak_; }

private:
    struct Block {
        void* p;
        int64_t bytes;
    };
    std::vector<Block> blocks_;
    hipStream_t stream_ = nullptr;
    int64_t budget_ = 0, bytes_ = 0, peak_ = 0;
    // fixed-region mode: a stack of block starts (offsets), no heap use
    static constexpr int REGION_STACK = 64;
    char* region_ = nullptr;
    int64_t capacity_ = 0, top_ = 0;
    bool fallback_ = false;
    int64_t starts_[REGION_STACK] = {};
    int nstarts_ = 0;
};

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline int bits_for(int64_t maxval) {  // bits needed to represent 0..maxval
    int b = 0;
    while (b < 63 && ((int64_t)1 << b) <= maxval) b++;
    return b;
}

// ---- primitives (prims.hip) ------------------------------------------------
// Exclusive prefix sum of n uint32 counts into uint64 offsets; out[n] = total
// when out has n+1 slots (write_total).  Temporary storage from `arena`.
void scan_u32_to_u64(const uint32_t* in, uint64_t* out, int64_t n, bool write_total, Arena& arena,
                     hipStream_t s);
// Same for int32 inputs into int64 outputs.
void scan_i32_to_i64(const int32_t* in, int64_t* out, int64_t n, bool write_total, Arena& arena,
                     hipStream_t s);
// Same for uint64 inputs.
void scan_u64(const uint64_t* in, uint64_t* out, int64_t n, bool write_total, Arena& arena, hipStream_t s);

// p[0..n) = v
void fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s);

// Stable LSD radix sort of 64-bit keys over bits [0, key_bits), carrying
// optional 32-bit values, ping-ponging between two caller buffers: the input
// is keys[cur] (vals[cur]); on return cur names the buffer holding the
// result.  An internal inconsistency sets bit `bad_bit` of *bad (device
// memory); the caller reads it at its next synchronisation.
template <class K>
struct SortBuffersT {
    K* keys[2];
    uint32_t* vals[2];  // both null when no values are carried
    int cur;
};
using SortBuffers = SortBuffersT<uint64_t>;
using SortBuffers32 = SortBuffersT<uint32_t>;
// first_hist (optional): counts of bits [0, 8) of the keys in each tile of
// RADIX_TILE keys, first_hist[tile * 256 + digit], written by the kernel
// that produced the keys; it replaces the first pass's histogram when that
// pass sorts an 8-bit digit.
constexpr int RADIX_TILE = 4096;
// first_bit: sort by bits [first_bit, first_bit + key_bits) only.
void radix_sort_u64(SortBuffers& b, int64_t n, int key_bits, Arena& arena, hipStream_t s, int* bad,
                    int bad_bit, uint32_t* first_hist = nullptr, int first_bit = 0);
// The same for 32-bit keys (key_bits <= 32): half the key traffic per pass.
void radix_sort_u32(SortBuffers32& b, int64_t n, int key_bits, Arena& arena, hipStream_t s, int* bad, int bad_bit);

// In-edges grouped by destination, sources ascending (sample.hip): built once
// per graph for the fanout sampler.  Complete when build_csc returns.
struct Csc {
    Arena arena;
    int64_t* in_off = nullptr;  // [n+1]
    int32_t* in_src = nullptr;  // [e]
    int32_t* heavy = nullptr;   // destinations with more than 64 in-edges
    int64_t nheavy = 0;
    double ms_build = 0;
    explicit Csc(hipStream_t s) : arena(s) {}
    // may be read from other streams than the one it was built on
    ~Csc() {
        (void)hipDeviceSynchronize();
        arena.set_stream(nullptr);
        arena.release();
    }
};
// scratch (optional): where the sort's temporaries go
std::shared_ptr<Csc> build_csc(const taurus_graph& g, hipStream_t s, Arena* scratch = nullptr);
// row_off monotone from 0 to e and col_dst in [0, n), else TAURUS_E_INVALID (synchronises)
void validate_csr(const taurus_graph& g, hipStream_t s);
// largest fanout a sampled layer takes
constexpr int FANOUT_MAX = 512;
// mask (device, ceil(e/64) words, CSR edge order) = the fanout-k sample of
// layer `layer`
void sample_mask(const taurus_graph& g, const Csc& csc, uint64_t seed, int layer, int k, uint64_t* mask,
                 hipStream_t s);
// The kept in-edges of the fanout-k sample as chunk-index items, in CSC
// order (destinations ascending, sources ascending within one): keys
// (chunk(u) << (vbits + 1) | nf << vbits | v) in sb.keys[0], nf = 1 when
// chunk(u) is after the earlier of v's own chunk and the chunk of v's
// smallest kept source (from key_arena, with its ping-pong
// buffer sb.keys[1]), values u - chunk(u)*C in sb.vals[0] (from val_arena,
// with sb.vals[1]).  Also m[v] = min(d_in(v), k) and first_chunk[v] = the
// chunk of v's smallest kept source (left as it was when none is kept).
// Returns the number kept.  Sets bit 32 of *bad (device) for an in-list
// the pass could not settle (repeated sources).
int64_t sample_items(const Csc& csc, int64_t n, uint64_t seed, int layer, int k, int64_t C, int vbits,
                     Arena& key_arena, Arena& val_arena, SortBuffers& sb, int32_t* m, int32_t* first_chunk, int* bad,
                     hipStream_t s);

}  // namespace taurus
