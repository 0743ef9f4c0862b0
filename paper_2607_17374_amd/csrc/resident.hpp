// Accumulator residency under a device-memory budget (resident.hip).
#pragma once

#include "internal.hpp"

namespace taurus {

constexpr int RES_LISTS = 6;  // the five short classes and the wave units of a chunk

// The destinations one chunk touches: its work units (v = unit.z) and its
// own vertices [first_row, first_row + rows) (the self message).
struct ResChunk {
    const int4* u[RES_LISTS];
    int64_t n[RES_LISTS];
    int64_t first_row, rows;
    int64_t total() const {
        int64_t t = rows;
        for (int l = 0; l < RES_LISTS; l++) t += n[l];
        return t;
    }
};

class Residency {
public:
    // slots: pool rows (hubs included); hubs: resident hub rows; m: message
    // counts per vertex (hub order); messages: their sum
    // policy: TAURUS_EVICT_*; seed: the random policy's; nchunks: the layer's chunk count
    Residency(hipStream_t s, int64_t n, int d_o, int64_t slots, int64_t hubs, const int32_t* m, int64_t messages,
              int policy, uint64_t seed, int64_t nchunks);
    ~Residency();
    Residency(const Residency&) = delete;
    Residency& operator=(const Residency&) = delete;

    // device bytes the residency structures take besides the pool
    static int64_t fixed_bytes(int64_t n);

    // give every pending destination of chunk k a slot, evicting if needed
    void prepare(const ResChunk& c, int32_t k, const int2* cnt, hipStream_t s);
    // free the slots of the chunk's destinations that completed
    void release(const ResChunk& c, const int2* cnt, hipStream_t s);
    int64_t reload_count(hipStream_t s);
    // counts[i] = vertices reloaded i times (i < bins - 1), counts[bins - 1] = the rest
    void reload_histogram(int64_t* counts, int bins, hipStream_t s);

    Arena arena;
    int64_t n, d_o, S, H;
    int policy;
    uint64_t seed;
    int chunk_shift = 0;
    float* pool = nullptr;       // [S][d_o]
    int32_t* slot_of = nullptr;  // [n], -1 = no row
    int64_t evictions = 0;
    double hub_share = 0;        // share of the layer's messages addressed to hubs

private:
    int32_t *dc_mark = nullptr, *want = nullptr, *tie = nullptr, *victims = nullptr, *need = nullptr;
    int32_t *adm = nullptr, *reloads_of = nullptr;
    int64_t* tie_rank = nullptr;
    uint8_t *hub = nullptr, *evicted = nullptr;
    unsigned int* hist = nullptr;
    unsigned long long* counters = nullptr;  // [0] listed, [1] victims, [2] reloads, [3] hub messages
    int32_t *free_list = nullptr, *free_top = nullptr;
    float* store_host = nullptr;  // pinned [n][d_o] (from the pinned block cache)
    size_t store_cap = 0;
    float* store_dev = nullptr;   // the same memory as seen by kernels
    // a lower bound of the free slots, kept on the host: a chunk that
    // touches at most this many destinations needs no eviction, so its slots
    // are assigned without reading anything back (releases only raise the
    // true count)
    int64_t free_lb = 0;
};

}  // namespace taurus
