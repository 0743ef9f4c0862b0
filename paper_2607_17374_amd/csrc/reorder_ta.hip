// Topology-aware reordering (Taurus, Sec. 3.8, Alg. 1) on the GPU.
//
// Positions r minimise the in-neighbourhood dispersion
//     J(r, mu) = sum_v 1/d(v) sum_{u in N(v)} (r(u) - mu(v))^2
// by alternating its closed-form minimisers
//     mu(v) = (1/d(v)) sum_{u in N(v)} r(u),
//     r(w)  = sum_{v : w in N(v)} mu(v)/d(v) / sum_{v : w in N(v)} 1/d(v),
// N(v) = v's in-neighbours plus v itself (every vertex aggregates a self
// message), d(v) = d_in(v) + 1; the sources of r(w) are w and its
// out-neighbours.  Alg. 1: r = pi0 once, then per update mu, r and
// pi = ArgSort(r) (ties by the lower ID), carrying r to the next update,
// until pi stops changing.
//
// Every update is three segmented sums over adjacency lists -- the centres
// over in-lists, the positions over CSR rows, the span and J of the new
// order over in-lists -- with fp64 values gathered by vertex.  Lists shorter
// than TA_HEAVY take 8 lanes each (a wave covers 8 consecutive vertices);
// longer ones are cut into pieces of TA_PIECE entries, one workgroup each,
// whose partial results the vertex's combine step adds in piece order.
// Summation order is fixed, so a run repeats bit for bit; it differs from a
// sequential sum, so positions agree with one within fp64 rounding.  The
// denominators of r depend on the graph only and are summed once per call.
// The ranking is a stable radix sort of r's bit pattern (r >= 0, so the bits
// sort like the values) with the vertex IDs as values.
//
// C(pi) and J(pi) of each order take the ranks as positions: per vertex the
// smallest and largest rank over N(v), and the exact integer sums
// s1 = sum rank, s2 = sum rank^2 (128-bit), so that
//     sum_{u in N(v)} (rank(u) - s1/d)^2 / d = (d*s2 - s1^2) / d^2
// is formed from an exact numerator.
#include <algorithm>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

namespace taurus {

namespace {

constexpr int TA_LANES = 8;        // lanes per short list
constexpr int64_t TA_HEAVY = 512;  // lists at least this long are cut into pieces
constexpr int64_t TA_PIECE = 2048; // entries per piece
constexpr int TA_BLOCK = 256;

typedef unsigned __int128 u128;

__host__ __device__ inline int64_t ceil_div_dev(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Heavy lists of one adjacency (CSR rows or in-lists): hrow[h] = vertex,
// pieces pstart[h] .. pstart[h+1]-1, prow[p] = h.
struct Heavy {
    int64_t H = 0, P = 0;
    int32_t* hrow = nullptr;
    int64_t* pstart = nullptr;
    int32_t* prow = nullptr;
};

__global__ void k_heavy_count(const int64_t* __restrict__ off, int64_t n, int32_t* __restrict__ is_heavy,
                              int32_t* __restrict__ pieces) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n) return;
    const int64_t d = off[v + 1] - off[v];
    const bool h = d >= TA_HEAVY;
    is_heavy[v] = h ? 1 : 0;
    pieces[v] = h ? (int32_t)ceil_div_dev(d, TA_PIECE) : 0;
}

__global__ void k_heavy_list(const int64_t* __restrict__ off, int64_t n, const int32_t* __restrict__ is_heavy,
                             const int64_t* __restrict__ hidx, const int64_t* __restrict__ pidx,
                             int32_t* __restrict__ hrow, int64_t* __restrict__ pstart, int32_t* __restrict__ prow,
                             int64_t P) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n || !is_heavy[v]) return;
    const int64_t h = hidx[v];
    hrow[h] = (int32_t)v;
    pstart[h] = pidx[v];
    const int64_t np = ceil_div_dev(off[v + 1] - off[v], TA_PIECE);
    for (int64_t j = 0; j < np; j++) prow[pidx[v] + j] = (int32_t)h;
    if (pidx[v] + np == P) pstart[h + 1] = P;  // the last heavy vertex closes the table
}

Heavy plan_heavy(const int64_t* off, int64_t n, Arena& arena, hipStream_t s) {
    Heavy hv;
    const unsigned gn = (unsigned)std::max<int64_t>(1, ceil_div(n, TA_BLOCK));
    Arena tmp(s);
    int32_t* flag = tmp.alloc<int32_t>(n, "heavy flags");
    int32_t* cnt = tmp.alloc<int32_t>(n, "piece counts");
    int64_t* hidx = tmp.alloc<int64_t>(n + 1, "heavy index");
    int64_t* pidx = tmp.alloc<int64_t>(n + 1, "piece index");
    k_heavy_count<<<gn, TA_BLOCK, 0, s>>>(off, n, flag, cnt);
    TAURUS_CHECK_LAUNCH();
    scan_i32_to_i64(flag, hidx, n, true, tmp, s);
    scan_i32_to_i64(cnt, pidx, n, true, tmp, s);
    {
        Readback rb;
        rb.add(&hv.H, hidx + n, 1);
        rb.add(&hv.P, pidx + n, 1);
        rb.run(s);
    }
    if (hv.H > 0) {
        hv.hrow = arena.alloc<int32_t>(hv.H, "heavy vertices");
        hv.pstart = arena.alloc<int64_t>(hv.H + 1, "heavy piece starts");
        hv.prow = arena.alloc<int32_t>(hv.P, "piece owners");
        k_heavy_list<<<gn, TA_BLOCK, 0, s>>>(off, n, flag, hidx, pidx, hv.hrow, hv.pstart, hv.prow, hv.P);
        TAURUS_CHECK_LAUNCH();
    }
    return hv;
}

// ---- fp64 segmented sums ---------------------------------------------------
// out(v) = finish(v, self[v] + sum_{k in list(v)} val[idx[k]]), with
//   MODE_CENTRE:   out = q[v] = (s / d) / d, d = list length + 1 (in-lists);
//   MODE_DENOM:    out = den[w] = s (CSR rows);
//   MODE_POSITION: out = r[w] = s / den[w], plus the sort key and ID.
enum { MODE_CENTRE = 0, MODE_DENOM = 1, MODE_POSITION = 2 };

struct SumOut {
    double* out;
    const double* den;
    uint64_t* keys;
    uint32_t* ids;
};

template <int MODE>
__device__ inline void finish_sum(int64_t v, int64_t len, double s, const SumOut& o) {
    if (MODE == MODE_CENTRE) {
        const double d = (double)(len + 1);
        o.out[v] = (s / d) / d;
    } else if (MODE == MODE_DENOM) {
        o.out[v] = s;
    } else {
        const double x = s / o.den[v];
        o.out[v] = x;
        o.keys[v] = (uint64_t)__double_as_longlong(x);
        o.ids[v] = (uint32_t)v;
    }
}

template <int MODE>
__global__ __launch_bounds__(TA_BLOCK) void k_sum_short(const int64_t* __restrict__ off,
                                                        const int32_t* __restrict__ idx, int64_t n,
                                                        const double* __restrict__ val, SumOut o) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t v = t / TA_LANES;
    const int sub = (int)(t % TA_LANES);
    int64_t a = 0, b = 0;
    if (v < n) {
        a = off[v];
        b = off[v + 1];
        if (b - a >= TA_HEAVY) b = a;  // the piece kernels take it
    }
    double s0 = 0.0, s1 = 0.0;
    int64_t k = a + sub;
    for (; k + TA_LANES < b; k += 2 * TA_LANES) {
        s0 += val[idx[k]];
        s1 += val[idx[k + TA_LANES]];
    }
    if (k < b) s0 += val[idx[k]];
    double s = s0 + s1;
#pragma unroll
    for (int m = TA_LANES / 2; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
    if (v < n && sub == 0 && off[v + 1] - a < TA_HEAVY) finish_sum<MODE>(v, b - a, val[v] + s, o);
}

// one workgroup per piece of a heavy list: partial[p] = sum over the piece
__global__ __launch_bounds__(TA_BLOCK) void k_sum_piece(const int64_t* __restrict__ off,
                                                        const int32_t* __restrict__ idx, Heavy hv,
                                                        const double* __restrict__ val,
                                                        double* __restrict__ partial) {
    __shared__ double part[TA_BLOCK / 64];
    const int64_t p = blockIdx.x;
    const int32_t h = hv.prow[p];
    const int32_t v = hv.hrow[h];
    const int64_t a = off[v] + (p - hv.pstart[h]) * TA_PIECE;
    const int64_t b = min(off[v + 1], a + TA_PIECE);
    double s0 = 0.0, s1 = 0.0;
    int64_t k = a + threadIdx.x;
    for (; k + TA_BLOCK < b; k += 2 * TA_BLOCK) {
        s0 += val[idx[k]];
        s1 += val[idx[k + TA_BLOCK]];
    }
    if (k < b) s0 += val[idx[k]];
    double s = s0 + s1;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = part[0];
        for (int w = 1; w < TA_BLOCK / 64; w++) t += part[w];
        partial[p] = t;
    }
}

// a thread per heavy list: own term plus the pieces in order
template <int MODE>
__global__ void k_sum_combine(const int64_t* __restrict__ off, Heavy hv, const double* __restrict__ val,
                              const double* __restrict__ partial, SumOut o) {
    const int64_t h = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (h >= hv.H) return;
    const int32_t v = hv.hrow[h];
    double s = 0.0;
    for (int64_t p = hv.pstart[h]; p < hv.pstart[h + 1]; p++) s += partial[p];
    finish_sum<MODE>(v, off[v + 1] - off[v], val[v] + s, o);
}

template <int MODE>
void seg_sum(const int64_t* off, const int32_t* idx, int64_t n, const Heavy& hv, const double* val,
             double* partial, const SumOut& o, hipStream_t s) {
    const int64_t threads = n * TA_LANES;
    k_sum_short<MODE><<<(unsigned)std::max<int64_t>(1, ceil_div(threads, TA_BLOCK)), TA_BLOCK, 0, s>>>(off, idx, n,
                                                                                                      val, o);
    TAURUS_CHECK_LAUNCH();
    if (hv.H > 0) {
        k_sum_piece<<<(unsigned)hv.P, TA_BLOCK, 0, s>>>(off, idx, hv, val, partial);
        TAURUS_CHECK_LAUNCH();
        k_sum_combine<MODE><<<(unsigned)ceil_div(hv.H, TA_BLOCK), TA_BLOCK, 0, s>>>(off, hv, val, partial, o);
        TAURUS_CHECK_LAUNCH();
    }
}

// ---- span and dispersion of an order ---------------------------------------
struct RankAcc {
    int32_t lo, hi;
    int64_t s1;
    u128 s2;
};

__device__ inline RankAcc rank_id() { return RankAcc{INT32_MAX, INT32_MIN, 0, 0}; }
__device__ inline void rank_add(RankAcc& a, int32_t p) {
    a.lo = min(a.lo, p);
    a.hi = max(a.hi, p);
    a.s1 += p;
    a.s2 += (u128)((uint64_t)p * (uint64_t)p);
}
__device__ inline void rank_merge(RankAcc& a, const RankAcc& b) {
    a.lo = min(a.lo, b.lo);
    a.hi = max(a.hi, b.hi);
    a.s1 += b.s1;
    a.s2 += b.s2;
}
__device__ inline RankAcc rank_shfl_xor(const RankAcc& a, int m) {
    RankAcc b;
    b.lo = __shfl_xor(a.lo, m, 64);
    b.hi = __shfl_xor(a.hi, m, 64);
    b.s1 = __shfl_xor(a.s1, m, 64);
    const uint64_t lo = __shfl_xor((uint64_t)a.s2, m, 64);
    const uint64_t hi = __shfl_xor((uint64_t)(a.s2 >> 64), m, 64);
    b.s2 = ((u128)hi << 64) | lo;
    return b;
}
__device__ inline double u128_to_f64(u128 x) {
    return (double)(uint64_t)(x >> 64) * 18446744073709551616.0 + (double)(uint64_t)x;
}
// span (max - min rank) and the dispersion term (d*s2 - s1^2) / d^2 of one
// neighbourhood of d members
__device__ inline void rank_terms(const RankAcc& a, int64_t d, int64_t& span, double& term) {
    span = (int64_t)a.hi - a.lo;
    const u128 s1 = (u128)(uint64_t)a.s1;
    const u128 num = (u128)(uint64_t)d * a.s2 - s1 * s1;
    term = u128_to_f64(num) / (double)d / (double)d;
}

__global__ __launch_bounds__(TA_BLOCK) void k_rank_short(const int64_t* __restrict__ off,
                                                         const int32_t* __restrict__ idx, int64_t n,
                                                         const int32_t* __restrict__ pi,
                                                         unsigned long long* __restrict__ span_total,
                                                         double* __restrict__ block_terms) {
    __shared__ double part[TA_BLOCK / 64];
    __shared__ unsigned long long spans;
    if (threadIdx.x == 0) spans = 0;
    __syncthreads();
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t v = t / TA_LANES;
    const int sub = (int)(t % TA_LANES);
    int64_t a = 0, b = 0;
    bool mine = false;
    if (v < n) {
        a = off[v];
        b = off[v + 1];
        mine = b - a < TA_HEAVY;
        if (!mine) b = a;
    }
    RankAcc acc = rank_id();
    for (int64_t k = a + sub; k < b; k += TA_LANES) rank_add(acc, pi[idx[k]]);
#pragma unroll
    for (int m = TA_LANES / 2; m >= 1; m >>= 1) rank_merge(acc, rank_shfl_xor(acc, m));
    double term = 0.0;
    if (mine && sub == 0) {
        rank_add(acc, pi[v]);
        int64_t sp;
        rank_terms(acc, b - a + 1, sp, term);
        if (sp) atomicAdd(&spans, (unsigned long long)sp);
    }
    // the block's terms in a fixed order: lanes 0, 8, ... of each wave, then waves
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) term += __shfl_xor(term, m, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = term;
    __syncthreads();
    if (threadIdx.x == 0) {
        double s = part[0];
        for (int w = 1; w < TA_BLOCK / 64; w++) s += part[w];
        block_terms[blockIdx.x] = s;
        if (spans) atomicAdd(span_total, spans);
    }
}

struct RankPart {
    int32_t lo, hi;
    int64_t s1;
    uint64_t s2lo, s2hi;
};

__global__ __launch_bounds__(TA_BLOCK) void k_rank_piece(const int64_t* __restrict__ off,
                                                         const int32_t* __restrict__ idx, Heavy hv,
                                                         const int32_t* __restrict__ pi,
                                                         RankPart* __restrict__ partial) {
    __shared__ RankPart part[TA_BLOCK / 64];
    const int64_t p = blockIdx.x;
    const int32_t h = hv.prow[p];
    const int32_t v = hv.hrow[h];
    const int64_t a = off[v] + (p - hv.pstart[h]) * TA_PIECE;
    const int64_t b = min(off[v + 1], a + TA_PIECE);
    RankAcc acc = rank_id();
    for (int64_t k = a + threadIdx.x; k < b; k += TA_BLOCK) rank_add(acc, pi[idx[k]]);
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) rank_merge(acc, rank_shfl_xor(acc, m));
    if ((threadIdx.x & 63) == 0)
        part[threadIdx.x >> 6] = RankPart{acc.lo, acc.hi, acc.s1, (uint64_t)acc.s2, (uint64_t)(acc.s2 >> 64)};
    __syncthreads();
    if (threadIdx.x == 0) {
        RankAcc t = rank_id();
        for (int w = 0; w < TA_BLOCK / 64; w++)
            rank_merge(t, RankAcc{part[w].lo, part[w].hi, part[w].s1, ((u128)part[w].s2hi << 64) | part[w].s2lo});
        partial[p] = RankPart{t.lo, t.hi, t.s1, (uint64_t)t.s2, (uint64_t)(t.s2 >> 64)};
    }
}

__global__ void k_rank_combine(const int64_t* __restrict__ off, Heavy hv, const int32_t* __restrict__ pi,
                               const RankPart* __restrict__ partial, unsigned long long* __restrict__ span_total,
                               double* __restrict__ heavy_terms) {
    const int64_t h = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (h >= hv.H) return;
    const int32_t v = hv.hrow[h];
    RankAcc acc = rank_id();
    rank_add(acc, pi[v]);
    for (int64_t p = hv.pstart[h]; p < hv.pstart[h + 1]; p++)
        rank_merge(acc, RankAcc{partial[p].lo, partial[p].hi, partial[p].s1,
                                ((u128)partial[p].s2hi << 64) | partial[p].s2lo});
    int64_t sp;
    double term;
    rank_terms(acc, off[v + 1] - off[v] + 1, sp, term);
    if (sp) atomicAdd(span_total, (unsigned long long)sp);
    heavy_terms[h] = term;
}

// one workgroup: J = the short blocks' sums, then the heavy terms, in order
__global__ __launch_bounds__(TA_BLOCK) void k_sum_terms(const double* __restrict__ a, int64_t na,
                                                        const double* __restrict__ b, int64_t nb,
                                                        double* __restrict__ out) {
    __shared__ double part[TA_BLOCK / 64];
    double s = 0.0;
    for (int64_t i = threadIdx.x; i < na; i += TA_BLOCK) s += a[i];
    for (int64_t i = threadIdx.x; i < nb; i += TA_BLOCK) s += b[i];
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) s += __shfl_xor(s, m, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = part[0];
        for (int w = 1; w < TA_BLOCK / 64; w++) t += part[w];
        *out = t;
    }
}

// ---- set-up, ranks ----------------------------------------------------------

// bootstrap: r = pi0 (the identity when pi0 is null), and a permutation check
__global__ void k_ta_init(const int32_t* __restrict__ pi0, int64_t n, double* __restrict__ r,
                          int32_t* __restrict__ pi, int32_t* __restrict__ seen, int* __restrict__ bad) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n) return;
    const int32_t p = pi0 ? pi0[v] : (int32_t)v;
    if (p < 0 || (int64_t)p >= n || atomicAdd(&seen[p], 1) != 0) atomicOr(bad, 1);
    r[v] = (double)p;
    pi[v] = p;
}

// 1/d(v) over the in-lists
__global__ void k_ta_inverse(const int64_t* __restrict__ in_off, int64_t n, double* __restrict__ inv) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n) inv[v] = 1.0 / (double)(in_off[v + 1] - in_off[v] + 1);
}

// new ranks from the sorted order; flags a vertex whose rank changed
__global__ void k_ta_ranks(const uint32_t* __restrict__ order, int64_t n, int32_t* __restrict__ pi,
                           int* __restrict__ changed) {
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= n) return;
    const uint32_t v = order[k];
    if (pi[v] != (int32_t)k) {
        pi[v] = (int32_t)k;
        atomicOr(changed, 1);
    }
}

}  // namespace

int reorder_ta_impl(const taurus_graph& g, const int32_t* pi0, int iters, int32_t* pi, double* positions,
                    int64_t* spans, double* disp, int32_t* done, hipStream_t s) {
    const int64_t n = g.n;
    const unsigned gn = (unsigned)std::max<int64_t>(1, ceil_div(n, TA_BLOCK));
    std::shared_ptr<Csc> csc = build_csc(g, s);  // validates the graph
    Arena tmp(s);
    const Heavy hin = plan_heavy(csc->in_off, n, tmp, s);
    const Heavy hout = plan_heavy(g.row_off, n, tmp, s);
    int* flags = tmp.alloc<int>(2, "flags");  // [0] bad bootstrap / changed, [1] sort
    unsigned long long* span = tmp.alloc<unsigned long long>(1, "span");
    double* jsum = tmp.alloc<double>(1, "dispersion");
    double* r = tmp.alloc<double>(n, "positions");
    double* q = tmp.alloc<double>(n, "centre terms");
    double* inv = tmp.alloc<double>(n, "inverse sizes");
    double* den = tmp.alloc<double>(n, "position denominators");
    const int64_t nparts = std::max<int64_t>(1, std::max(hin.P, hout.P));
    double* partial = tmp.alloc<double>(nparts, "piece sums");
    RankPart* rpart = tmp.alloc<RankPart>(std::max<int64_t>(1, hin.P), "piece ranks");
    const int64_t nshort = std::max<int64_t>(1, ceil_div(n * TA_LANES, TA_BLOCK));
    double* block_terms = tmp.alloc<double>(nshort, "dispersion block sums");
    double* heavy_terms = tmp.alloc<double>(std::max<int64_t>(1, hin.H), "dispersion heavy terms");
    int32_t* seen = tmp.alloc<int32_t>(n, "bootstrap marks");
    SortBuffers sb{{tmp.alloc<uint64_t>(n, "position keys"), tmp.alloc<uint64_t>(n, "position keys (ping-pong)")},
                   {tmp.alloc<uint32_t>(n, "order"), tmp.alloc<uint32_t>(n, "order (ping-pong)")},
                   0};
    // C(pi) and J(pi) of the current order; reads them back with the flags
    auto measure = [&](int* flag_out, double* j_out) {
        fill_i32(reinterpret_cast<int32_t*>(span), 2, 0, s);
        k_rank_short<<<(unsigned)nshort, TA_BLOCK, 0, s>>>(csc->in_off, csc->in_src, n, pi, span, block_terms);
        TAURUS_CHECK_LAUNCH();
        if (hin.H > 0) {
            k_rank_piece<<<(unsigned)hin.P, TA_BLOCK, 0, s>>>(csc->in_off, csc->in_src, hin, pi, rpart);
            TAURUS_CHECK_LAUNCH();
            k_rank_combine<<<(unsigned)ceil_div(hin.H, TA_BLOCK), TA_BLOCK, 0, s>>>(csc->in_off, hin, pi, rpart, span,
                                                                                 heavy_terms);
            TAURUS_CHECK_LAUNCH();
        }
        k_sum_terms<<<1, TA_BLOCK, 0, s>>>(block_terms, n > 0 ? nshort : 0, heavy_terms, hin.H, jsum);
        TAURUS_CHECK_LAUNCH();
        unsigned long long c = 0;
        int f[2] = {0, 0};
        Readback rb;
        rb.add(&c, span, 1);
        rb.add(j_out, jsum, 1);
        rb.add(f, flags, 2);
        rb.run(s);
        if (flag_out) *flag_out = f[0];
        if (f[1]) fail(TAURUS_E_DEVICE, "reorder: radix sort offset out of range");
        return (int64_t)c;
    };
    fill_i32(flags, 2, 0, s);
    fill_i32(seen, n, 0, s);
    k_ta_init<<<gn, TA_BLOCK, 0, s>>>(pi0, n, r, pi, seen, flags);
    TAURUS_CHECK_LAUNCH();
    k_ta_inverse<<<gn, TA_BLOCK, 0, s>>>(csc->in_off, n, inv);
    TAURUS_CHECK_LAUNCH();
    // the denominators of r: 1/d over w and its out-neighbours
    seg_sum<MODE_DENOM>(g.row_off, g.col_dst, n, hout, inv, partial, SumOut{den, nullptr, nullptr, nullptr}, s);
    int bad = 0;
    double j0 = 0.0;
    const int64_t c0 = measure(&bad, &j0);
    if (bad) fail(TAURUS_E_INVALID, "bootstrap order is not a permutation of [0, n)");
    if (spans) spans[0] = c0;
    if (disp) disp[0] = j0;
    *done = 0;
    for (int t = 1; t <= iters; t++) {
        seg_sum<MODE_CENTRE>(csc->in_off, csc->in_src, n, hin, r, partial, SumOut{q, nullptr, nullptr, nullptr}, s);
        sb.cur = 0;
        seg_sum<MODE_POSITION>(g.row_off, g.col_dst, n, hout, q, partial, SumOut{r, den, sb.keys[0], sb.vals[0]},
                               s);
        radix_sort_u64(sb, n, 64, tmp, s, flags + 1, 1);
        fill_i32(flags, 1, 0, s);
        k_ta_ranks<<<gn, TA_BLOCK, 0, s>>>(sb.vals[sb.cur], n, pi, flags);
        TAURUS_CHECK_LAUNCH();
        int changed = 0;
        double jt = 0.0;
        const int64_t c = measure(&changed, &jt);
        if (spans) spans[t] = c;
        if (disp) disp[t] = jt;
        *done = t;
        if (!changed) break;
    }
    if (positions && n > 0) TAURUS_HIP(hipMemcpyAsync(positions, r, (size_t)n * sizeof(double), hipMemcpyDeviceToDevice, s));
    TAURUS_HIP(hipStreamSynchronize(s));
    return TAURUS_OK;
}

}  // namespace taurus
