// Search-based vertex orderings (topology-aware bootstraps in the sense of
// Sec. 3.8: a destination's sources get nearby ranks, which shrinks the span
// between its first and last message) and relabelling.
//
// Both orderings are the visit order of a sequential breadth-first search
// whose roots and children are ranked by a degree key, ties by lower ID:
//   - degree/BFS: search over in-edges (vertex -> its in-neighbours), key
//     in-degree descending;
//   - RCMK (reverse Cuthill-McKee, the bootstrap Sec. 3.8 names): search
//     over the symmetrised graph, key symmetric degree ascending, and the
//     visit order reversed.
// Every root not yet visited starts a search, and a dequeued vertex appends
// its unvisited neighbours in key order.
//
// The GPU computes exactly that order without a queue:
//   1. rank[v] = position of v in the root order (radix sort);
//   2. owner[v] = min rank over every vertex v can reach along the reverse
//      of the search's lists (out-edges for the in-edge search, the
//      symmetric lists themselves for RCMK; v itself included): the search
//      started by the root of rank r visits exactly the vertices with owner
//      r, because a vertex belongs to the first root it can reach.  Computed
//      by min-label propagation over the edges plus a shortcut through each
//      label's own root, to a fixed point;
//   3. trees are laid out one after another in root order (a histogram of
//      owners and a scan give each tree's offset), roots take the first slot
//      of their tree;
//   4. all trees advance one level at a time: every unvisited vertex w on
//      the list of a frontier vertex x in w's own tree is claimed by the frontier
//      vertex with the smallest position (the first one the queue would
//      dequeue); the new level is sorted by (claimer's position, rank[w]) --
//      the order the queue appends them in -- and takes the next free slots
//      of its tree.
#include "device.hpp"
#include "internal.hpp"

namespace taurus {

int build_csr_impl(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                   int32_t* col_dst, hipStream_t s);

// root-order key: d << idbits | v (degree ascending) or (n-1 - d) << idbits | v
// (degree descending), ID ascending either way; d = deg_off[v+1] - deg_off[v] <= n-1
__global__ void k_root_keys(const int64_t* __restrict__ deg_off, int64_t n, int idbits, int ascending,
                            uint64_t* __restrict__ keys, uint32_t* __restrict__ vals) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n) return;
    const int64_t d = deg_off[v + 1] - deg_off[v];
    keys[v] = ((uint64_t)(ascending ? d : n - 1 - d) << idbits) | (uint64_t)v;
    vals[v] = (uint32_t)v;
}

// order[r] = the vertex of rank r (the sorted values); rank[order[r]] = r
__global__ void k_ranks(const uint32_t* __restrict__ order, int64_t n, int32_t* __restrict__ rank,
                        int32_t* __restrict__ label) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= n) return;
    const uint32_t v = order[r];
    rank[v] = (int32_t)r;
    label[v] = (int32_t)r;
}

// label[u] = min(label[u], label[v]) over edges (u, v): u reaches all v
// reaches.  A workgroup takes LE_TILE consecutive edges (rows found through
// tile_rows), 64 consecutive ones per wave at a time; edges of one row are
// contiguous, so each wave reduces runs of equal u with shuffles first and
// issues one atomic per run.
constexpr int LE_ITEMS = 16, LE_TILE = 256 * LE_ITEMS, LE_ROWS = 8192;
__global__ __launch_bounds__(256) void k_label_edges(const int64_t* __restrict__ row_off,
                                                     const int32_t* __restrict__ col_dst, int64_t n, int64_t e,
                                                     int32_t* __restrict__ label, int* __restrict__ changed) {
    __shared__ int32_t ro[LE_ROWS + 1];
    __shared__ int64_t bnd[2];
    const int lane = threadIdx.x & 63;
    const int64_t i0 = (int64_t)blockIdx.x * LE_TILE, i1 = min(i0 + LE_TILE, e);
    const TileRows t = tile_rows<LE_ROWS, LE_TILE>(row_off, n, i0, i1, ro, bnd);
    bool any = false;
    for (int r = 0; r < LE_ITEMS; r++) {
        if (i0 + (int64_t)r * 256 >= i1) break;  // uniform over the workgroup
        const int64_t i = i0 + (int64_t)r * 256 + threadIdx.x;
        const bool valid = i < i1;
        bool later;
        const int64_t u = valid ? tile_row_of(t, row_off, ro, i0, i, later) : -1;
        int32_t m = valid ? label[col_dst[i]] : INT32_MAX;
        // inclusive segmented minimum over lanes with the same u
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const int32_t om = __shfl_up(m, d, 64);
            const int64_t ou = __shfl_up(u, d, 64);
            if (lane >= d && ou == u) m = min(m, om);
        }
        const int64_t nu = __shfl_down(u, 1, 64);
        const bool next_valid = __shfl_down((int)valid, 1, 64) != 0;
        const bool last = valid && (lane == 63 || !next_valid || nu != u);
        if (last && m < label[u]) {
            atomicMin(&label[u], m);
            any = true;
        }
    }
    if (any) *changed = 1;
}

// shortcut: v reaches the root of rank label[v], hence everything that root
// reaches: label[v] = min(label[v], label[order[label[v]]])
__global__ void k_label_jump(const uint32_t* __restrict__ order, int64_t n, int32_t* __restrict__ label,
                             int* __restrict__ changed) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n) return;
    const int32_t l = label[v];
    const int32_t l2 = label[order[l]];
    if (l2 < l) {
        atomicMin(&label[v], l2);
        *changed = 1;
    }
}

// size[l] = vertices labelled l.  Lanes of a wave with the same label add
// once (a giant component would otherwise put nearly every vertex's atomic
// on one counter): the first remaining lane's label is matched by ballot,
// that lane adds the matches, and the rest go round again.
__global__ void k_tree_sizes(const int32_t* __restrict__ label, int64_t n, int32_t* __restrict__ size) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int lane = threadIdx.x & 63;
    const int32_t l = v < n ? label[v] : -1;
    uint64_t left = __ballot(v < n);
    while (left) {  // uniform over the wave
        const int lead = __builtin_ctzll(left);
        const int32_t ll = __shfl(l, lead);
        const uint64_t same = __ballot(v < n && l == ll);
        if (lane == lead) atomicAdd(&size[ll], (int)__popcll(same));
        left &= ~same;
    }
}

// roots: pos = the first slot of their tree; they form the first frontier
__global__ void k_roots(const int32_t* __restrict__ label, const int32_t* __restrict__ rank,
                        const int64_t* __restrict__ off, int64_t n, int32_t* __restrict__ pos,
                        int32_t* __restrict__ next, int32_t* __restrict__ frontier,
                        unsigned long long* __restrict__ count) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n) return;
    const int32_t r = rank[v];
    const bool root = label[v] == r;
    if (root) {
        pos[v] = (int32_t)off[r];
        next[r] = 1;
    }
    const unsigned long long at = wave_append(root, count);
    if (root) frontier[at] = (int32_t)v;
}

// One wave per frontier vertex x: each unvisited neighbour w (x's search
// list) in x's tree records the smallest claiming position and is listed once.
__global__ __launch_bounds__(256) void k_expand(const int32_t* __restrict__ frontier, int64_t nf,
                                                const int64_t* __restrict__ in_off,
                                                const int32_t* __restrict__ in_src,
                                                const int32_t* __restrict__ label, const int32_t* __restrict__ pos,
                                                int32_t* __restrict__ claim, int32_t* __restrict__ listed,
                                                int32_t* __restrict__ cand, unsigned long long* __restrict__ count) {
    const int lane = threadIdx.x & 63;
    const int64_t f = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (f >= nf) return;
    const int32_t x = frontier[f];
    const int32_t px = pos[x], lx = label[x];
    for (int64_t k = in_off[x] + lane; k < in_off[x + 1]; k += 64) {
        const int32_t w = in_src[k];
        bool add = false;
        if (pos[w] < 0 && label[w] == lx) {
            atomicMin(&claim[w], px);
            add = atomicExch(&listed[w], 1) == 0;
        }
        const unsigned long long at = wave_append(add, count);
        if (add) cand[at] = w;
    }
}

// key (claiming position, rank): the order the queue appends the level in
__global__ void k_level_keys(const int32_t* __restrict__ cand, int64_t nc, const int32_t* __restrict__ claim,
                             const int32_t* __restrict__ rank, int rbits, uint64_t* __restrict__ keys,
                             uint32_t* __restrict__ vals) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= nc) return;
    const int32_t w = cand[j];
    keys[j] = ((uint64_t)claim[w] << rbits) | (uint64_t)rank[w];
    vals[j] = (uint32_t)w;
}

// first index of each tree's run in the sorted level
__global__ void k_level_heads(const uint32_t* __restrict__ sorted, int64_t nc, const int32_t* __restrict__ label,
                              int32_t* __restrict__ start) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= nc) return;
    const int32_t t = label[sorted[j]];
    if (j == 0 || label[sorted[j - 1]] != t) start[t] = (int32_t)j;
}

__global__ void k_level_assign(const uint32_t* __restrict__ sorted, int64_t nc, const int32_t* __restrict__ label,
                               const int64_t* __restrict__ off, const int32_t* __restrict__ next,
                               const int32_t* __restrict__ start, int32_t* __restrict__ pos,
                               int32_t* __restrict__ frontier) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= nc) return;
    const int32_t w = (int32_t)sorted[j];
    const int32_t t = label[w];
    pos[w] = (int32_t)(off[t] + next[t] + (j - start[t]));
    frontier[j] = w;
}

// after the positions are written: each tree's next free slot moves past its run
__global__ void k_level_advance(const uint32_t* __restrict__ sorted, int64_t nc, const int32_t* __restrict__ label,
                                const int32_t* __restrict__ start, int32_t* __restrict__ next) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= nc) return;
    const int32_t t = label[sorted[j]];
    if (j == nc - 1 || label[sorted[j + 1]] != t) next[t] += (int32_t)(j - start[t] + 1);
}

__global__ void k_flag(const int32_t* __restrict__ pos, int64_t n, int* __restrict__ bad) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n && (pos[v] < 0 || pos[v] >= n)) atomicOr(bad, 1);
}

__global__ void k_reverse(int32_t* __restrict__ pos, int64_t n) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v < n) pos[v] = (int32_t)(n - 1 - pos[v]);
}

// The lists a search walks and the graph its owners come from.
struct Search {
    const int64_t* reach_off;  // owner labels: u reaches reach_adj[reach_off[u] .. reach_off[u+1])
    const int32_t* reach_adj;
    int64_t reach_e;
    const int64_t* list_off;  // a dequeued x appends from list_adj[list_off[x] .. list_off[x+1]);
    const int32_t* list_adj;  // its length is the degree of the key
    bool ascending;           // key: degree ascending (else descending), then ID ascending
    bool reverse;             // new_of_old = n - 1 - visit position
};

static void search_order(int64_t n, const Search& sp, int32_t* new_of_old, hipStream_t s) {
    const int64_t e = sp.reach_e;
    const int T = 256;
    auto blocks = [&](int64_t count) { return (unsigned)std::max<int64_t>(1, ceil_div(count, T)); };
    Arena tmp(s);
    const int idbits = std::max(1, bits_for(n - 1));
    int* flag = tmp.alloc<int>(2, "flags");  // [0] changed, [1] sort/consistency

    // 1. root order
    SortBuffers rs{{tmp.alloc<uint64_t>(n, "root keys"), tmp.alloc<uint64_t>(n, "root keys (ping-pong)")},
                   {tmp.alloc<uint32_t>(n, "root order"), tmp.alloc<uint32_t>(n, "root order (ping-pong)")},
                   0};
    k_root_keys<<<blocks(n), T, 0, s>>>(sp.list_off, n, idbits, sp.ascending ? 1 : 0, rs.keys[0], rs.vals[0]);
    TAURUS_CHECK_LAUNCH();
    fill_i32(flag, 2, 0, s);
    radix_sort_u64(rs, n, 2 * idbits, tmp, s, flag + 1, 1);
    const uint32_t* order = rs.vals[rs.cur];
    int32_t* rank = tmp.alloc<int32_t>(n, "root ranks");
    int32_t* label = tmp.alloc<int32_t>(n, "owners");
    k_ranks<<<blocks(n), T, 0, s>>>(order, n, rank, label);
    TAURUS_CHECK_LAUNCH();

    // 2. owners, to a fixed point
    for (int iter = 0;; iter++) {
        if (iter > 4 * n + 8) fail(TAURUS_E_DEVICE, "reorder: owner labels did not converge");
        fill_i32(flag, 1, 0, s);
        if (e > 0) {
            k_label_edges<<<(unsigned)ceil_div(e, LE_TILE), T, 0, s>>>(sp.reach_off, sp.reach_adj, n, e, label, flag);
            TAURUS_CHECK_LAUNCH();
        }
        k_label_jump<<<blocks(n), T, 0, s>>>(order, n, label, flag);
        TAURUS_CHECK_LAUNCH();
        int changed = 0;
        Readback rb;
        rb.add(&changed, flag, 1);
        rb.run(s);
        if (!changed) break;
    }

    // 3. tree offsets, roots
    int32_t* size = tmp.alloc<int32_t>(n, "tree sizes");
    fill_i32(size, n, 0, s);
    k_tree_sizes<<<blocks(n), T, 0, s>>>(label, n, size);
    TAURUS_CHECK_LAUNCH();
    int64_t* off = tmp.alloc<int64_t>(n + 1, "tree offsets");
    scan_i32_to_i64(size, off, n, true, tmp, s);
    int32_t* pos = new_of_old;
    fill_i32(pos, n, -1, s);
    int32_t* next = tmp.alloc<int32_t>(n, "next free slot per tree");
    fill_i32(next, n, 0, s);
    int32_t* claim = tmp.alloc<int32_t>(n, "claiming positions");
    fill_i32(claim, n, INT32_MAX, s);
    int32_t* listed = tmp.alloc<int32_t>(n, "listed flags");
    fill_i32(listed, n, 0, s);
    int32_t* start = tmp.alloc<int32_t>(n, "run starts");
    int32_t* frontier = tmp.alloc<int32_t>(n, "frontier");
    int32_t* cand = tmp.alloc<int32_t>(n, "candidates");
    unsigned long long* count = tmp.alloc<unsigned long long>(1, "count");
    fill_i32(reinterpret_cast<int32_t*>(count), 2, 0, s);
    k_roots<<<blocks(n), T, 0, s>>>(label, rank, off, n, pos, next, frontier, count);
    TAURUS_CHECK_LAUNCH();
    unsigned long long nf = 0;
    {
        Readback rb;
        rb.add(&nf, count, 1);
        rb.run(s);
    }
    SortBuffers ls{{tmp.alloc<uint64_t>(n, "level keys"), tmp.alloc<uint64_t>(n, "level keys (ping-pong)")},
                   {tmp.alloc<uint32_t>(n, "level vertices"), tmp.alloc<uint32_t>(n, "level vertices (ping-pong)")},
                   0};
    const int pbits = std::max(1, bits_for(n - 1));

    // 4. levels
    int64_t visited = (int64_t)nf;
    while (nf > 0) {
        fill_i32(reinterpret_cast<int32_t*>(count), 2, 0, s);
        k_expand<<<(unsigned)ceil_div((int64_t)nf * 64, T), T, 0, s>>>(frontier, (int64_t)nf, sp.list_off,
                                                                     sp.list_adj, label, pos, claim, listed,
                                                                     cand, count);
        TAURUS_CHECK_LAUNCH();
        unsigned long long nc = 0;
        {
            Readback rb;
            rb.add(&nc, count, 1);
            rb.run(s);
        }
        if (nc == 0) break;
        if ((int64_t)nc > n - visited) fail(TAURUS_E_DEVICE, "reorder: more candidates than unvisited vertices");
        ls.cur = 0;
        k_level_keys<<<blocks((int64_t)nc), T, 0, s>>>(cand, (int64_t)nc, claim, rank, idbits, ls.keys[0],
                                                       ls.vals[0]);
        TAURUS_CHECK_LAUNCH();
        radix_sort_u64(ls, (int64_t)nc, pbits + idbits, tmp, s, flag + 1, 1);
        const uint32_t* sorted = ls.vals[ls.cur];
        k_level_heads<<<blocks((int64_t)nc), T, 0, s>>>(sorted, (int64_t)nc, label, start);
        TAURUS_CHECK_LAUNCH();
        k_level_assign<<<blocks((int64_t)nc), T, 0, s>>>(sorted, (int64_t)nc, label, off, next, start, pos,
                                                         frontier);
        TAURUS_CHECK_LAUNCH();
        k_level_advance<<<blocks((int64_t)nc), T, 0, s>>>(sorted, (int64_t)nc, label, start, next);
        TAURUS_CHECK_LAUNCH();
        nf = nc;
        visited += (int64_t)nc;
    }
    k_flag<<<blocks(n), T, 0, s>>>(pos, n, flag + 1);
    TAURUS_CHECK_LAUNCH();
    int bad = 0;
    {
        Readback rb;
        rb.add(&bad, flag + 1, 1);
        rb.run(s);
    }
    if (bad || visited != n) fail(TAURUS_E_DEVICE, "reorder: %lld of %lld vertices placed", (long long)visited,
                                  (long long)n);
    if (sp.reverse) {
        k_reverse<<<blocks(n), T, 0, s>>>(pos, n);
        TAURUS_CHECK_LAUNCH();
    }
}

int reorder_impl(const taurus_graph& g, int32_t* new_of_old, hipStream_t s) {
    std::shared_ptr<Csc> csc = build_csc(g, s);  // validates the graph
    const Search sp{g.row_off, g.col_dst, g.e, csc->in_off, csc->in_src, false, false};
    search_order(g.n, sp, new_of_old, s);
    return TAURUS_OK;
}

// ---------------------------------------------------------------- RCMK -----
// Per CSR edge (u, v): miss[i] = 1 when (v, u) is not an edge (binary search
// of u in v's strictly ascending row).
__global__ __launch_bounds__(256) void k_sym_missing(const int64_t* __restrict__ row_off,
                                                     const int32_t* __restrict__ col_dst, int64_t n, int64_t e,
                                                     uint32_t* __restrict__ miss) {
    __shared__ int64_t ro[4][64];
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t u = wave_edge_row(row_off, n, i, ro[threadIdx.x >> 6]);
    if (i >= e) return;
    const int32_t v = col_dst[i];
    int64_t lo = row_off[v], hi = row_off[v + 1];
    while (lo < hi) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (col_dst[mid] < u) lo = mid + 1;
        else hi = mid;
    }
    miss[i] = (lo < row_off[v + 1] && col_dst[lo] == u) ? 0u : 1u;
}

// the symmetric pair list: every edge (u, v), then (v, u) for each edge whose
// reverse is missing, at e + (its rank among those)
__global__ __launch_bounds__(256) void k_sym_pairs(const int64_t* __restrict__ row_off,
                                                   const int32_t* __restrict__ col_dst, int64_t n, int64_t e,
                                                   const uint32_t* __restrict__ miss,
                                                   const uint64_t* __restrict__ miss_rank,
                                                   int32_t* __restrict__ src, int32_t* __restrict__ dst) {
    __shared__ int64_t ro[4][64];
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t u = wave_edge_row(row_off, n, i, ro[threadIdx.x >> 6]);
    if (i >= e) return;
    const int32_t v = col_dst[i];
    src[i] = (int32_t)u;
    dst[i] = v;
    if (miss[i]) {
        const int64_t j = e + (int64_t)miss_rank[i];
        src[j] = v;
        dst[j] = (int32_t)u;
    }
}

int reorder_rcm_impl(const taurus_graph& g, int32_t* new_of_old, hipStream_t s) {
    validate_csr(g, s);
    const int64_t n = g.n, e = g.e;
    const int T = 256;
    Arena sym(s);
    int64_t* sym_off = sym.alloc<int64_t>(n + 1, "symmetric offsets");
    int32_t* sym_adj = nullptr;
    int64_t es = 0;
    if (e > 0) {
        Arena pairs(s);
        int32_t *src = nullptr, *dst = nullptr;
        {
            Arena tmp(s);
            uint32_t* miss = tmp.alloc<uint32_t>(e, "missing reverse flags");
            uint64_t* rank = tmp.alloc<uint64_t>(e + 1, "missing reverse ranks");
            k_sym_missing<<<(unsigned)ceil_div(e, T), T, 0, s>>>(g.row_off, g.col_dst, n, e, miss);
            TAURUS_CHECK_LAUNCH();
            scan_u32_to_u64(miss, rank, e, true, tmp, s);
            uint64_t m = 0;
            Readback rb;
            rb.add(&m, rank + e, 1);
            rb.run(s);
            es = e + (int64_t)m;
            src = pairs.alloc<int32_t>(es, "symmetric sources");
            dst = pairs.alloc<int32_t>(es, "symmetric destinations");
            k_sym_pairs<<<(unsigned)ceil_div(e, T), T, 0, s>>>(g.row_off, g.col_dst, n, e, miss, rank, src, dst);
            TAURUS_CHECK_LAUNCH();
        }
        sym_adj = sym.alloc<int32_t>(es, "symmetric lists");
        build_csr_impl(n, es, src, dst, sym_off, sym_adj, s);  // sorted, no repeats, no self loops
    } else {
        fill_i32(reinterpret_cast<int32_t*>(sym_off), 2 * (n + 1), 0, s);
    }
    const Search sp{sym_off, sym_adj, es, sym_off, sym_adj, true, true};
    search_order(n, sp, new_of_old, s);
    return TAURUS_OK;
}

// ------------------------------------------------------------- relabel -----
// edge i of the CSR in the new numbering; LE_TILE edges per workgroup, rows
// found through tile_rows
__global__ __launch_bounds__(256) void k_relabel_edges(const int64_t* __restrict__ row_off,
                                                       const int32_t* __restrict__ col_dst, int64_t n, int64_t e,
                                                       const int32_t* __restrict__ new_of_old,
                                                       int32_t* __restrict__ src, int32_t* __restrict__ dst) {
    __shared__ int32_t ro[LE_ROWS + 1];
    __shared__ int64_t bnd[2];
    const int64_t i0 = (int64_t)blockIdx.x * LE_TILE, i1 = min(i0 + LE_TILE, e);
    const TileRows t = tile_rows<LE_ROWS, LE_TILE>(row_off, n, i0, i1, ro, bnd);
#pragma unroll 4
    for (int r = 0; r < LE_ITEMS; r++) {
        const int64_t i = i0 + (int64_t)r * 256 + threadIdx.x;
        if (i >= i1) break;
        bool later;
        const int64_t u = tile_row_of(t, row_off, ro, i0, i, later);
        src[i] = new_of_old[u];
        dst[i] = new_of_old[col_dst[i]];
    }
}

__global__ void k_check_perm(const int32_t* __restrict__ p, int64_t n, int32_t* __restrict__ seen,
                             int* __restrict__ bad) {
    const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (v >= n) return;
    const int32_t x = p[v];
    if (x < 0 || x >= n || atomicExch(&seen[x], 1) != 0) atomicOr(bad, 1);
}

static void check_permutation(const int32_t* p, int64_t n, Arena& tmp, hipStream_t s) {
    int32_t* seen = tmp.alloc<int32_t>(n, "permutation check");
    fill_i32(seen, n, 0, s);
    int* bad = tmp.alloc<int>(1, "permutation flag");
    fill_i32(bad, 1, 0, s);
    k_check_perm<<<(unsigned)ceil_div(n, 256), 256, 0, s>>>(p, n, seen, bad);
    TAURUS_CHECK_LAUNCH();
    int hbad = 0;
    Readback rb;
    rb.add(&hbad, bad, 1);
    rb.run(s);
    if (hbad) fail(TAURUS_E_INVALID, "new_of_old is not a permutation of [0, n)");
}

int relabel_impl(const taurus_graph& g, const int32_t* new_of_old, int64_t* row_off, int32_t* col_dst,
                 hipStream_t s) {
    validate_csr(g, s);  // the graph is walked below
    Arena tmp(s);
    check_permutation(new_of_old, g.n, tmp, s);
    int32_t* src = tmp.alloc<int32_t>(std::max<int64_t>(1, g.e), "relabelled sources");
    int32_t* dst = tmp.alloc<int32_t>(std::max<int64_t>(1, g.e), "relabelled destinations");
    if (g.e > 0) {
        k_relabel_edges<<<(unsigned)ceil_div(g.e, LE_TILE), 256, 0, s>>>(g.row_off, g.col_dst, g.n, g.e, new_of_old,
                                                                         src, dst);
        TAURUS_CHECK_LAUNCH();
    }
    return build_csr_impl(g.n, g.e, src, dst, row_off, col_dst, s);
}

// one wave per row; rows of 16-byte words when row_bytes % 16 == 0, else of
// 4-byte words
template <typename W>
__global__ __launch_bounds__(256) void k_permute_rows(const W* __restrict__ in, W* __restrict__ out, int64_t n,
                                                      int64_t words, const int32_t* __restrict__ new_of_old,
                                                      int inverse) {
    const int64_t v = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (v >= n) return;
    const int64_t p = new_of_old[v];
    const W* a = in + (inverse ? p : v) * words;
    W* b = out + (inverse ? v : p) * words;
    for (int64_t w = threadIdx.x & 63; w < words; w += 64) b[w] = a[w];
}

int permute_rows_impl(const void* in, void* out, int64_t n, int64_t row_bytes, const int32_t* new_of_old,
                      int inverse, hipStream_t s) {
    Arena tmp(s);
    check_permutation(new_of_old, n, tmp, s);
    const unsigned grid = (unsigned)ceil_div(n * 64, 256);
    if (row_bytes % 16 == 0)
        k_permute_rows<uint4><<<grid, 256, 0, s>>>(static_cast<const uint4*>(in), static_cast<uint4*>(out), n,
                                                   row_bytes / 16, new_of_old, inverse);
    else
        k_permute_rows<uint32_t><<<grid, 256, 0, s>>>(static_cast<const uint32_t*>(in), static_cast<uint32_t*>(out),
                                                      n, row_bytes / 4, new_of_old, inverse);
    TAURUS_CHECK_LAUNCH();
    return TAURUS_OK;
}

}  // namespace taurus
