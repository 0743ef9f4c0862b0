// Device helpers shared by the kernel files: the sampler's hash, wave
// appends, searches for the CSR row of an edge, the chunk index's per-vertex
// flags and output-row stores.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace taurus {

// Per-vertex flags of a layer's chunk index.
constexpr uint8_t OWN_SEGMENT = 1;  // v has a segment from its own chunk
constexpr uint8_t SELF_FIRST = 2;   // no message to v comes from an earlier chunk

// fp32 to bf16 bits, round to nearest even (a NaN stays a quiet NaN)
__device__ inline uint32_t f32_to_bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}
__device__ inline uint32_t f32_to_f16_bits(float f) {
    const _Float16 h = (_Float16)f;  // v_cvt_f16_f32, round to nearest even
    return (uint32_t)__builtin_bit_cast(uint16_t, h);
}

// Four consecutive output values at element idx of out, stored as dtype
// (0 fp32, 1 bf16, 2 fp16).
__device__ inline void store_out4(void* out, int dtype, int64_t idx, float4 z) {
    if (dtype == 0) {
        *reinterpret_cast<float4*>(static_cast<float*>(out) + idx) = z;
    } else {
        uint2 p;
        if (dtype == 1) {
            p.x = f32_to_bf16_bits(z.x) | (f32_to_bf16_bits(z.y) << 16);
            p.y = f32_to_bf16_bits(z.z) | (f32_to_bf16_bits(z.w) << 16);
        } else {
            p.x = f32_to_f16_bits(z.x) | (f32_to_f16_bits(z.y) << 16);
            p.y = f32_to_f16_bits(z.z) | (f32_to_f16_bits(z.w) << 16);
        }
        *reinterpret_cast<uint2*>(static_cast<uint16_t*>(out) + idx) = p;
    }
}

// SplitMix64 finaliser and increment (Steele, Lea and Flood, OOPSLA 2014).
constexpr uint64_t SM64_GAMMA = 0x9e3779b97f4a7c15ULL;

__host__ __device__ inline uint64_t mix64(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

// Sampling rank hash H(seed, 4, layer, v, u): the counter hash chained over
// the tag and arguments (h = mix64(h + gamma + x) for each), split so that
// the per-destination prefix H(seed, 4, layer, v) is computed once.
__host__ __device__ inline uint64_t sample_prefix(uint64_t seed, uint64_t layer, uint64_t v) {
    uint64_t h = mix64(seed + SM64_GAMMA + 4u);
    h = mix64(h + SM64_GAMMA + layer);
    return mix64(h + SM64_GAMMA + v);
}
__host__ __device__ inline uint64_t sample_key(uint64_t prefix, uint64_t u) { return mix64(prefix + SM64_GAMMA + u); }

// Slot in a list of length *count for each lane that appends one entry
// (want): the wave's appending lanes take consecutive slots with a single
// atomic, so a list that grows by millions of entries does not serialise on
// its counter.  Lanes that do not append get 0 and must ignore it.  Call from
// every active lane that may append.
template <class C>
__device__ inline C wave_append(bool want, C* count) {
    const uint64_t b = __ballot(want);
    if (!b) return 0;
    const int lane = threadIdx.x & 63;
    const int lead = __builtin_ctzll(b);
    C base = 0;
    if (lane == lead) base = atomicAdd(count, (C)__popcll(b));
    base = __shfl(base, lead);
    return base + (C)__popcll(b & ((1ull << lane) - 1ull));
}

// Row of CSR edge t for a whole wave (every lane passes the same t): the
// largest u in [0, n) with row_off[u] <= t, by a 64-ary search (every lane
// probes at once, ~log64(n) dependent loads).  All probes stay in [0, n].
// Every lane of the wave must call it (it uses ballots).
__device__ inline int64_t wave_row_of(const int64_t* __restrict__ row_off, int64_t n, int64_t t) {
    const int lane = threadIdx.x & 63;
    int64_t lo = 0, hi = n;
    while (hi - lo > 64) {
        const int64_t step = (hi - lo + 63) >> 6;
        const int64_t p = min(lo + (int64_t)(lane + 1) * step, hi);
        const int k = __popcll(__ballot(row_off[p] <= t));
        const int64_t nlo = lo + (int64_t)k * step;
        hi = min(nlo + step, hi);
        lo = nlo;
    }
    {
        const int64_t p = lo + lane + 1;
        const int k = __popcll(__ballot(p <= hi && row_off[p] <= t));
        lo += k;
    }
    return min(lo, n - 1);
}

// Rows of a workgroup's tile of CSR edges [i0, i1) (i0 < i1 <= e), for
// kernels that take TILE consecutive edges per workgroup: two waves find the
// rows ua and ub of the first and last edge (wave_row_of); when the tile
// spans at most ROWS rows, their starts go to `ro` in LDS (relative to i0,
// clamped to [-1, TILE + 1]) and each edge finds its row there by binary
// search, else (many empty rows) by binary search of row_off between ua and
// ub.  (Finding each thread's first row once and walking forward over its
// consecutive edges, recorded per edge in LDS, measured slower.)  Memory
// safe on invalid offsets (rows stay in [0, n)).  Called by the whole
// workgroup (it has barriers); `ro` holds ROWS + 1 entries.
struct TileRows {
    int64_t ua, ub, nr;
    bool staged;
};
template <int ROWS, int TILE>
__device__ inline TileRows tile_rows(const int64_t* __restrict__ row_off, int64_t n, int64_t i0, int64_t i1,
                                     int32_t* ro, int64_t* bnd) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (wave < 2) {
        const int64_t u = wave_row_of(row_off, n, wave == 0 ? i0 : i1 - 1);
        if (lane == 0) bnd[wave] = u;
    }
    __syncthreads();
    TileRows t;
    t.ua = bnd[0];
    t.ub = bnd[1];
    t.nr = t.ub - t.ua + 1;
    t.staged = t.nr >= 1 && t.nr <= ROWS;
    if (t.staged)
        for (int64_t j = threadIdx.x; j <= t.nr; j += blockDim.x) {  // j = nr: the end of the last row
            const int64_t x = row_off[t.ua + j] - i0;
            ro[j] = (int32_t)max(min(x, (int64_t)TILE + 1), (int64_t)-1);
        }
    __syncthreads();
    return t;
}
// Row of edge i of the tile; `later`: i is not the first edge of its row.
__device__ inline int64_t tile_row_of(const TileRows& t, const int64_t* __restrict__ row_off, const int32_t* ro,
                                      int64_t i0, int64_t i, bool& later) {
    if (t.staged) {
        const int32_t li = (int32_t)(i - i0);
        int a = 0, z = (int)t.nr;  // the last row start at or before li
        while (z - a > 1) {
            const int mid = (a + z) >> 1;
            if (ro[mid] <= li) a = mid;
            else z = mid;
        }
        later = ro[a] < li && i > 0;
        return t.ua + a;
    }
    int64_t a = t.ua, z = max(t.ub + 1, t.ua + 1);
    while (z - a > 1) {
        const int64_t mid = (a + z) >> 1;
        if (row_off[mid] <= i) a = mid;
        else z = mid;
    }
    later = i > row_off[a];
    return a;
}

// Row (source) of CSR edge i = lane's edge, for all 64 lanes of a wave whose
// first edge is i0 = i - lane.  The wave finds the row u0 of i0 with a 64-ary
// search (every lane probes at once, ~log64(n) dependent loads instead of
// ~log2(n) per lane), stages row_off[u0+1 .. u0+64] in `ro` (64 entries of
// LDS owned by the wave), and each lane locates its own edge among those; an
// edge more than 64 rows past u0 (only after many empty rows) falls back to
// a binary search of the rest.  All probes stay in [0, n], also for lanes
// with i >= e and for invalid offsets; the result is in [0, n).  Every lane
// of the wave must call it (it uses ballots and a wave-level barrier between
// its LDS writes and reads).
__device__ inline int64_t wave_edge_row(const int64_t* __restrict__ row_off, int64_t n, int64_t i,
                                        int64_t* ro) {
    const int lane = threadIdx.x & 63;
    const int64_t u0 = wave_row_of(row_off, n, i - lane);
    const int64_t q = u0 + 1 + lane;
    ro[lane] = q <= n ? row_off[q] : INT64_MAX;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    if (ro[63] <= i) {
        int64_t a = u0 + 64, z = n;  // largest u in [a, n) with row_off[u] <= i
        while (z - a > 1) {
            const int64_t mid = (a + z) >> 1;
            if (row_off[mid] <= i) a = mid;
            else z = mid;
        }
        return min(a, n - 1);
    }
    int c = 0;
#pragma unroll
    for (int half = 32; half >= 1; half >>= 1)
        if (ro[c + half - 1] <= i) c += half;
    return u0 + c;
}

}  // namespace taurus
