// Topology-aware reordering (Taurus, Sec. 3.8, Alg. 1) on the GPU.
//
// Positions r minimise the in-neighbourhood dispersion
//     J(r, mu) = sum_v 1/d(v) sum_{u in N(v)} (r(u) - mu(v))^2
// with its closed-form minimisers
//     mu(v) = (1/d(v)) sum_{u in N(v)} r(u),
//     r(w)  = sum_{v : w in N(v)} mu(v)/d(v) / sum_{v : w in N(v)} 1/d(v),
// and ranks the vertices by r.  N(v) is v's propagated in-neighbours plus v
// itself (every vertex aggregates a self message), d(v) = d_in(v) + 1, so the
// sources of r(w) are w and its out-neighbours.  Each update starts from the
// current order as the positions (r = pi), so an order that an update leaves
// unchanged is a fixed point and stopping there is exact.
//
// Every sum runs in fp64 in one fixed order, the vertex's own term first and
// then its neighbours in ascending ID (a thread per vertex walking its
// in-list or CSR row), so the positions are the same bit for bit on every
// run and on any machine that follows that order.  The ranking is a stable
// radix sort of r's bit pattern (r >= 0, so the bits sort like the values)
// with the vertex IDs as values: ties go to the lower ID.
#include <algorithm>
#include <vector>

#include "device.hpp"
#include "internal.hpp"

namespace taurus {

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

// mu(v), and the terms a destination v gives the positions of its sources:
// q(v) = mu(v) / d(v) and inv(v) = 1 / d(v)
__global__ void k_ta_centres(const int64_t* __restrict__ in_off, const int32_t* __restrict__ in_src, int64_t n,
                             const double* __restrict__ r, double* __restrict__ q, double* __restrict__ inv) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n) return;
    const int64_t a = in_off[v], b = in_off[v + 1];
    double s = r[v];
    for (int64_t k = a; k < b; k++) s += r[in_src[k]];
    const double d = (double)(b - a + 1);
    const double mu = s / d;
    q[v] = mu / d;
    inv[v] = 1.0 / d;
}

// r(w) over w and its out-neighbours; the sort key is r's bit pattern
__global__ void k_ta_positions(const int64_t* __restrict__ row_off, const int32_t* __restrict__ col_dst, int64_t n,
                               const double* __restrict__ q, const double* __restrict__ inv, double* __restrict__ r,
                               uint64_t* __restrict__ keys, uint32_t* __restrict__ ids) {
    const int64_t w = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (w >= n) return;
    double num = q[w], den = inv[w];
    for (int64_t i = row_off[w]; i < row_off[w + 1]; i++) {
        const int32_t v = col_dst[i];
        num += q[v];
        den += inv[v];
    }
    const double x = num / den;
    r[w] = x;
    keys[w] = (uint64_t)__double_as_longlong(x);
    ids[w] = (uint32_t)w;
}

// new_of_old from the sorted order, and the next update's positions r = pi;
// flags a vertex whose rank changed
__global__ void k_ta_ranks(const uint32_t* __restrict__ order, int64_t n, int32_t* __restrict__ pi,
                           double* __restrict__ r, int* __restrict__ changed) {
    const int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= n) return;
    const uint32_t v = order[k];
    r[v] = (double)k;
    if (pi[v] != (int32_t)k) {
        pi[v] = (int32_t)k;
        atomicOr(changed, 1);
    }
}

// C(pi) = sum over vertices of (max - min) rank over the vertex and its
// propagated in-neighbours (the total span of Sec. 3.8, self message included)
__global__ __launch_bounds__(256) void k_total_span(const int64_t* __restrict__ in_off,
                                                    const int32_t* __restrict__ in_src, int64_t n,
                                                    const int32_t* __restrict__ pi,
                                                    unsigned long long* __restrict__ total) {
    __shared__ unsigned long long part;
    if (threadIdx.x == 0) part = 0;
    __syncthreads();
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n && in_off[v + 1] > in_off[v]) {
        int32_t lo = pi[v], hi = pi[v];
        for (int64_t k = in_off[v]; k < in_off[v + 1]; k++) {
            const int32_t p = pi[in_src[k]];
            lo = min(lo, p);
            hi = max(hi, p);
        }
        atomicAdd(&part, (unsigned long long)(hi - lo));
    }
    __syncthreads();
    if (threadIdx.x == 0 && part) atomicAdd(total, part);
}

int reorder_ta_impl(const taurus_graph& g, const int32_t* pi0, int iters, int32_t* pi, int64_t* spans,
                    int32_t* done, hipStream_t s) {
    const int64_t n = g.n;
    const int T = 256;
    const unsigned gn = (unsigned)std::max<int64_t>(1, ceil_div(n, T));
    std::shared_ptr<Csc> csc = build_csc(g, s);  // validates the graph
    Arena tmp(s);
    int* flags = tmp.alloc<int>(2, "flags");                    // [0] bad bootstrap / changed, [1] sort
    unsigned long long* span = tmp.alloc<unsigned long long>(1, "span");
    double* r = tmp.alloc<double>(n, "positions");
    double* q = tmp.alloc<double>(n, "centre terms");
    double* inv = tmp.alloc<double>(n, "inverse sizes");
    int32_t* seen = tmp.alloc<int32_t>(n, "bootstrap marks");
    SortBuffers sb{{tmp.alloc<uint64_t>(n, "position keys"), tmp.alloc<uint64_t>(n, "position keys (ping-pong)")},
                   {tmp.alloc<uint32_t>(n, "order"), tmp.alloc<uint32_t>(n, "order (ping-pong)")},
                   0};
    auto read_span = [&](int* flag_out) {
        fill_i32(reinterpret_cast<int32_t*>(span), 2, 0, s);
        k_total_span<<<gn, T, 0, s>>>(csc->in_off, csc->in_src, n, pi, span);
        TAURUS_CHECK_LAUNCH();
        unsigned long long c = 0;
        int f[2] = {0, 0};
        Readback rb;
        rb.add(&c, span, 1);
        rb.add(f, flags, 2);
        rb.run(s);
        if (flag_out) *flag_out = f[0];
        if (f[1]) fail(TAURUS_E_DEVICE, "reorder: radix sort offset out of range");
        return (int64_t)c;
    };
    fill_i32(flags, 2, 0, s);
    fill_i32(seen, n, 0, s);
    k_ta_init<<<gn, T, 0, s>>>(pi0, n, r, pi, seen, flags);
    TAURUS_CHECK_LAUNCH();
    int bad = 0;
    const int64_t c0 = read_span(&bad);
    if (bad) fail(TAURUS_E_INVALID, "bootstrap order is not a permutation of [0, n)");
    if (spans) spans[0] = c0;
    *done = 0;
    for (int t = 1; t <= iters; t++) {
        k_ta_centres<<<gn, T, 0, s>>>(csc->in_off, csc->in_src, n, r, q, inv);
        TAURUS_CHECK_LAUNCH();
        sb.cur = 0;
        k_ta_positions<<<gn, T, 0, s>>>(g.row_off, g.col_dst, n, q, inv, r, sb.keys[0], sb.vals[0]);
        TAURUS_CHECK_LAUNCH();
        radix_sort_u64(sb, n, 64, tmp, s, flags + 1, 1);
        fill_i32(flags, 1, 0, s);
        k_ta_ranks<<<gn, T, 0, s>>>(sb.vals[sb.cur], n, pi, r, flags);
        TAURUS_CHECK_LAUNCH();
        int changed = 0;
        const int64_t c = read_span(&changed);
        if (spans) spans[t] = c;
        *done = t;
        if (!changed) break;
    }
    return TAURUS_OK;
}

}  // namespace taurus
