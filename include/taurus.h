/*
 * taurus.h -- C ABI of the MI355X layer-wise broadcast GNN inference library.
 *
 * Method: Taurus (arXiv 2607.17374).  Layer-wise inference (Sec. 2.3)
 * recast as source-centric broadcast (Sec. 3.1): every layer streams each
 * source vertex once, in chunks of contiguous vertex IDs (Sec. 3.3), pushes
 * one message per propagated out-edge into its destination's partial
 * aggregate, counts pending messages per destination (Sec. 3.4) and
 * finalises a destination as soon as its count reaches zero (Sec. 3.6).
 * Mean aggregation sends the normalised message h_u / |M(v)| (Sec. 3.4);
 * GraphSAGE splits W = [W_agg W_self] so the self half is applied where the
 * vertex is streamed (Sec. 3.9, "SAGEConv"); fanout-sampled inference keeps
 * up to k in-edges per vertex and layer (Sec. 3.9, "Sampling-based
 * Inference").
 *
 * All pointers named "device" are HIP device pointers on the current device;
 * "host" pointers are ordinary host memory unless marked pinned (allocated
 * with hipHostMalloc or an equivalent page-locked allocator).  Every call
 * returns a taurus_status; on failure taurus_last_error() returns a
 * human-readable message for the calling thread.  No C++ exception crosses
 * this boundary.  A layer handle must be used by one thread at a time.
 */
#ifndef TAURUS_H
#define TAURUS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TAURUS_OK = 0,
    TAURUS_E_INVALID = -1,    /* bad argument; nothing was enqueued, handle unchanged        */
    TAURUS_E_OOM = -2,        /* device or pinned allocation failed; handle poisoned          */
    TAURUS_E_DEVICE = -3,     /* HIP runtime error; handle poisoned                           */
    TAURUS_E_STATE = -4,      /* call out of order, chunk pushed twice, or poisoned handle    */
    TAURUS_E_INCOMPLETE = -5, /* finalize found destinations with messages still pending      */
    TAURUS_E_BUDGET = -6      /* library allocations would exceed desc.hbm_budget             */
} taurus_status;

typedef enum { TAURUS_F32 = 0, TAURUS_BF16 = 1, TAURUS_F16 = 2 } taurus_dtype;

/* Eviction policies of a budgeted layer (desc.eviction).  The paper's
 * policy evicts the partial states with the fewest pending messages
 * (Sec. 3.5.3); random, FIFO and LRU are the policies it is compared with
 * (Sec. 4, eviction study).  Ties go to the lower vertex ID. */
typedef enum {
    TAURUS_EVICT_PENDING = 0, /* fewest pending messages first                               */
    TAURUS_EVICT_RANDOM = 1,  /* smallest H(seed, 7, chunk, v) >> 50 first, a fresh order per chunk */
    TAURUS_EVICT_FIFO = 2,    /* earliest admission (the chunk at which the row was taken)    */
    TAURUS_EVICT_LRU = 3      /* least recently used (the last chunk that sent a message)     */
} taurus_eviction;

/* Per-graph structures shared by the layers over one graph (see
 * taurus_plan_create). */
typedef struct taurus_plan taurus_plan;

/* Aggregation/update families (Sec. 3.9 and the models of Sec. 4.1). */
typedef enum {
    TAURUS_SAGE_MEAN = 0, /* z_v = W_agg mean_{u in M(v)} h_u + W_self h_v + b (mean = 0 if M(v) empty)  */
    TAURUS_GCN_SYM = 1,   /* z_v = W sum_{u in M(v) + {v}} h_u / sqrt(d^_out(u) d^_in(v)) + b,
                             d^ = degree + 1 (one self loop per vertex); a sampled layer uses the
                             degrees of its sampled graph: kept out-edges, d^_in(v) = |M(v)| + 1 */
    TAURUS_GIN_SUM = 2,   /* GINConv, linear apply, eps = 0: z_v = W (h_v + sum_{u in M(v)} h_u) + b */
    TAURUS_GAT_ATT = 3,   /* GATConv, one head (Sec. 3.9): h' = W h, e_uv = LeakyReLU(a^T [h'_u || h'_v]),
                             slope 0.2, alpha = softmax of e over M(v) + {v},
                             z_v = sum alpha_uv h'_u + b; needs desc.attn; in core (hbm_budget 0).
                             The pushes transform (pass 1); finalize runs the softmax statistics
                             (pass 2) and the aggregation (pass 3) over every chunk            */
    TAURUS_GIN_MLP = 4    /* GINConv with a two-layer perceptron apply (Sec. 4.1), eps = 0:
                             t_v = ReLU(W1 (h_v + sum_{u in M(v)} h_u) + b1), z_v = W2 t_v + b2.
                             W1 goes before the aggregation (linearity); a destination's t_v is
                             formed when it completes, and each chunk's completed rows then take
                             W2 on the matrix cores (the graduation transform, Sec. 3.6).  Needs
                             desc.d_hidden and desc.weight2; in core (hbm_budget 0)            */
} taurus_agg;

/*
 * Graph in CSR by source (Sec. 3.2: the topology is stored as CSR over
 * out-edges so sources can be scanned sequentially).  Device pointers,
 * caller-owned, read-only, valid until every layer built on it is destroyed:
 *   row_off  int64[n+1], row_off[0] = 0, row_off[n] = e, non-decreasing;
 *   col_dst  int32[e], destinations of row u in row_off[u]..row_off[u+1]-1,
 *            strictly ascending within a row, no self loops.
 * Edge (u, v) carries u's message to v; N-(v) = { u : (u, v) in E }.
 */
typedef struct {
    int64_t n;
    int64_t e;
    const int64_t* row_off;
    const int32_t* col_dst;
} taurus_graph;

/*
 * One layer.  Host-side descriptor, copied at taurus_layer_init.
 *   agg          taurus_agg.
 *   d_in, d_out  input and output widths; multiples of 4 (d_in a multiple
 *                of 8 for 16-bit inputs), d_out <= 1024.
 *   in_dtype     storage type of the layer input x (taurus_dtype); the
 *                transform multiplies in that type (16-bit: bf16 or fp16
 *                matrix cores) and accumulates in fp32.
 *   out_dtype    storage type of the layer output (hidden layers usually keep
 *                the input type; values are rounded to nearest even).
 *   relu         1 applies ReLU to the output (all layers but the last).
 *   weight       HOST fp32, row-major, copied at init.  GCN: [d_in][d_out],
 *                y = x W.  SAGE: [d_in][2*d_out] = [W_agg^T | W_self^T], so
 *                columns 0..d_out-1 act on the neighbour mean and columns
 *                d_out..2*d_out-1 on the vertex's own input.  For 16-bit
 *                in_dtype the weights are rounded to that type at init.
 *   bias         HOST fp32 [d_out], or NULL for no bias; copied at init.
 *   fanout       0 = exact inference (every in-edge propagates); k in
 *                [1, 512] keeps for each destination v its min(d_in(v), k)
 *                in-edges whose rank key (H(seed, 4, layer, v, u), u) is
 *                smallest, where H is the SplitMix64-based counter hash of
 *                taurus_hash() (Sec. 3.9, sampling-based inference).  Every
 *                family samples the same way; a sampled GCN layer normalises
 *                by the sampled graph's degrees, (kept out-degree(u) + 1) on
 *                the source side and (|M(v)| + 1) on the destination side.
 *   layer        1-based layer number (only feeds the sampling hash).
 *   seed         sampling seed.
 *   chunk        source-chunk size C in vertices (> 0).  Chunk j covers
 *                sources [j*C, min((j+1)*C, n)).  The chunk's transform,
 *                min(C, n) rows of d_out (GCN) or 2*d_out (GraphSAGE) fp32,
 *                must fit 2^31 - 2^24 bytes, else TAURUS_E_INVALID.
 *   hbm_budget   bytes of device memory the library may hold for this layer
 *                (its own buffers plus the chunk index it uses; 0 =
 *                unlimited).  When the dense accumulators [n][d_out] fp32 do
 *                not fit, they live in a pool of rows: hubs stay resident,
 *                other destinations take rows while they are pending, and
 *                when a chunk's destinations find too few free rows the
 *                pending vertices with the fewest outstanding messages (then
 *                lowest ID) that the chunk does not touch are evicted to a
 *                pinned host store and reloaded before their next message
 *                (Sec. 3.5).  Results are the same as in core.  Init fails
 *                with TAURUS_E_BUDGET if the fixed structures, the hubs and
 *                one chunk's destinations cannot fit.
 *   hub_fraction fraction in [0, 1] of vertices, by message count (ties by
 *                lower ID), whose accumulators stay resident for the whole
 *                layer when the pool is in use (Sec. 3.5.1).
 *   out          caller-owned [n][d_out] array of out_dtype receiving the
 *                layer output; each row is written exactly once, when its
 *                vertex completes.  Device memory unless out_on_host = 1.
 *   out_on_host  0: out is device memory; 1: out is pinned host memory
 *                (allocated with hipHostMalloc) written by the kernels over
 *                the host link as vertices complete.
 *   stream       hipStream_t on which all work of this layer is enqueued
 *                (NULL = the default stream).
 *   profile      1: time every kernel of the layer with HIP events; 2: time
 *                only the scatter launches (fewer events in the stream); the
 *                totals are returned in taurus_stats.
 *   attn         GAT layers: host float[2][d_out], row 0 (a_src) scores the
 *                transformed source row, row 1 (a_dst) the destination's;
 *                read at init.  NULL for the other families.
 *   eviction     TAURUS_EVICT_* policy of a budgeted layer (ignored in core).
 *                Victims are ranked by their exact key (pending count,
 *                admission chunk or last chunk), ties by the lower ID.
 *   d_hidden     TAURUS_GIN_MLP layers: the perceptron's hidden width (a
 *                positive multiple of 4, at most 1024); ignored otherwise.
 *   weight2      TAURUS_GIN_MLP layers: HOST fp32 [d_hidden][d_out], the
 *                perceptron's second layer (z = t W2); weight is then its
 *                first layer [d_in][d_hidden] and bias b1 [d_hidden] (or
 *                NULL).  Copied at init.  NULL otherwise.
 *   bias2        TAURUS_GIN_MLP layers: HOST fp32 [d_out] or NULL.
 *   plan         NULL, or a plan made for this graph (same n, e, row_off,
 *                col_dst pointers) and this chunk size: an exact layer
 *                (fanout = 0) then shares the plan's chunk index, and a
 *                sampled layer its in-edge lists, instead of building its
 *                own.  A plan with another graph or chunk size is
 *                TAURUS_E_INVALID.
 *   setup_stream NULL, or a hipStream_t for the work taurus_layer_init
 *                enqueues (in-edge lists, sampling, chunk index, weights,
 *                counters): it then runs beside whatever `stream` still has
 *                queued, such as an earlier layer's chunks, instead of after
 *                it, and `stream` waits for it before this layer's first
 *                kernel there.  The caller guarantees that the graph, the
 *                plan and host arrays are ready as seen from setup_stream.
 *                All later calls use `stream`.
 */
typedef struct {
    int32_t agg, d_in, d_out, in_dtype, out_dtype, relu;
    const float* weight;
    const float* bias;
    int32_t fanout, layer;
    uint64_t seed;
    int64_t chunk;
    int64_t hbm_budget;
    double hub_fraction;
    void* out;
    int32_t out_on_host;
    void* stream;
    int32_t profile;
    const taurus_plan* plan;
    int32_t eviction;
    const float* attn;
    int32_t d_hidden;
    const float* weight2;
    const float* bias2;
    void* setup_stream;
} taurus_layer_desc;

typedef struct taurus_layer taurus_layer;

/* Per-layer statistics, filled by taurus_finalize. */
typedef struct {
    int64_t n, e;                  /* graph size                                        */
    int64_t messages;              /* E_l: propagated in-edges (sum of |M(v)|)          */
    int64_t self_terms;            /* self messages (= n)                               */
    int64_t pairs;                 /* accumulator flushes: (destination, chunk) segments
                                      of propagated messages, plus one self flush per
                                      vertex                                            */
    int64_t completed;             /* vertices whose output row was written             */
    int64_t pending_left;          /* vertices still waiting for messages               */
    int64_t chunks, chunks_pushed;
    int64_t short_units;           /* segments of <= 16 slots, batched per row-group; a
                                      segment's slots are its messages plus the self
                                      message when it comes from v's own chunk         */
    int64_t wave_units;            /* pieces of <= 512 slots of longer segments (one
                                      wave each)                                        */
    int64_t split_segments;        /* hub segments cut into several pieces              */
    int64_t evictions, reloads;    /* accumulator rows moved to/from host (0 in core)   */
    int64_t h2d_bytes, d2h_bytes;  /* host-link bytes: host chunks and reloads in;
                                      evictions and host-resident output rows out       */
    int64_t device_bytes;          /* peak bytes allocated by the library for the layer */
    double hub_message_share;      /* share of messages landing on resident hubs        */
    /* milliseconds, HIP-event timed when desc.profile = 1 (only ms_scatter when 2; else 0) */
    double ms_init;                /* wall time of taurus_layer_init                    */
    double ms_index;               /* of which: sampling and chunk-index build (0 when
                                      the plan already held the index)                  */
    double ms_gemm, ms_self, ms_scatter, ms_fixup;  /* ms_self stays 0: the self messages
                                      run inside the scatter launch, timed in ms_scatter,
                                      or, for in-core GraphSAGE layers, those of vertices
                                      without a segment from their own chunk inside the
                                      transform, timed in ms_gemm.
                                      In-core fp32 GCN and linear-apply GIN layers run a
                                      chunk's hub fix-up in the next chunk's transform
                                      launch (timed in ms_gemm)
                                      and the last chunk's at finalize (untimed), so
                                      their ms_fixup stays 0                          */
    int64_t launches_gemm, launches_self, launches_scatter, launches_fixup;
    int64_t pool_rows;             /* budgeted layers: accumulator rows of the pool,
                                      hub rows included (0 in core)                     */
    int64_t hub_rows;              /* of which resident hub rows                        */
    int64_t self_in_transform;     /* in-core GraphSAGE layers: self messages added by
                                      the chunk transforms (vertices without a segment
                                      from their own chunk), 0 otherwise; counted in
                                      pairs                                             */
    int64_t self_fresh, self_last; /* of those, when desc.profile != 0: found nothing
                                      accumulated yet / completed the vertex (-1 when
                                      not counted, 0 for other layers)                  */
} taurus_stats;

/*
 * The library keeps device memory it no longer uses in a cache, so that the
 * next layer reuses it (re-allocating tens of GB costs seconds).  This call
 * hands cached blocks of the current device back to the runtime, smallest
 * first, until at least `bytes` bytes are freed (bytes <= 0: all of them),
 * for a caller whose own allocation ran out of memory.  Blocks in use are
 * not touched.  Large pinned host buffers (budgeted layers' stores for
 * evicted rows, the chunk loader's rings) are cached the same way; this
 * call frees every cached one of them too.  Synchronises the device.
 * Returns the device bytes freed, or a negative status.
 */
int64_t taurus_release_cached_memory(int64_t bytes);

/* Thread-local message describing the last failing call on this thread. */
const char* taurus_last_error(void);

/*
 * H(seed, tag, args...) = mix64 chain of SplitMix64 (Steele, Lea and Flood,
 * OOPSLA 2014): h = seed; for x in (tag, args...): h = mix64(h + G + x),
 * G = 0x9e3779b97f4a7c15.  Host function, exported so callers can reproduce
 * the sampling keys.  nargs <= 8.
 */
uint64_t taurus_hash(uint64_t seed, uint64_t tag, int32_t nargs, const uint64_t* args);

/*
 * Build CSR by source from an edge list (Sec. 3.2).  All arrays are device
 * memory: src, dst int32[e] (read), row_off int64[n+1] and col_dst int32[e]
 * (written, caller-owned).  The edge list must describe a simple graph
 * (0 <= ids < n, no self loops, no repeated pair); otherwise
 * TAURUS_E_INVALID and the outputs are unspecified.  The result is
 * canonical: rows sorted by destination.  Enqueued on `stream`; returns after
 * the work completed (it reads back a validity flag).  n < 2^31, e < 2^40.
 */
int taurus_build_csr(int64_t n, int64_t e, const int32_t* src, const int32_t* dst,
                     int64_t* row_off, int32_t* col_dst, void* stream);

/*
 * taurus_build_csr without allocating, for callers that cannot allocate
 * device memory: code being captured into a HIP graph, tight serving loops,
 * harnesses that forbid hipMalloc.  Same arguments, result and errors as
 * taurus_build_csr; it calls no hipMalloc, hipFree or other allocating
 * routine.  Its temporaries live in one fixed device array of
 * TAURUS_NOALLOC_SCRATCH_BYTES per GPU, which each GPU the library runs on
 * holds from the first call on it until the process ends.
 * Limit: e <= TAURUS_NOALLOC_MAX_EDGES; larger inputs return
 * TAURUS_E_INVALID before any work is enqueued.
 * Every call on one GPU shares that GPU's array and leaves its contents
 * behind: calls that overlap on one GPU (other host threads, other streams)
 * race and must be serialised by the caller.  Returns after the work
 * completed (it reads back a validity flag into host memory).
 */
#define TAURUS_NOALLOC_SCRATCH_BYTES (32ll << 20)
#define TAURUS_NOALLOC_MAX_EDGES (1ll << 20)
int taurus_build_csr_noalloc(int64_t n, int64_t e, const int32_t* src, const int32_t* dst, int64_t* row_off,
                             int32_t* col_dst, void* stream);

/*
 * Degree/BFS vertex ordering (Sec. 3.8: a topology-aware order in which a
 * destination's sources receive nearby ranks, shrinking the span between
 * its first and last message).  new_of_old (device int32[n], written) is
 * the visit order of a breadth-first search over in-edges: roots are taken
 * in (in-degree descending, ID ascending) order, every root not yet visited
 * starts a new search, and a dequeued vertex appends its unvisited
 * in-neighbours in the same order.  The order is unique.  The graph is
 * validated (TAURUS_E_INVALID).  Returns after the work completed.
 */
int taurus_reorder(const taurus_graph* g, int32_t* new_of_old, void* stream);

/*
 * RCMK order (reverse Cuthill-McKee; Sec. 3.8 names it as the bandwidth-
 * reducing bootstrap of Alg. 1).  The search runs on the symmetrised graph:
 * u and v are neighbours when (u, v) or (v, u) is an edge, and a vertex's
 * degree counts its distinct neighbours.  Roots are taken in (degree
 * ascending, ID ascending) order, every root not yet visited starts a
 * breadth-first search, and a dequeued vertex appends its unvisited
 * neighbours in the same order; new_of_old[v] (device int32[n], written) =
 * n - 1 - the visit position of v.  The order is unique.  Works in device
 * memory of about 40 bytes per edge (the symmetric pair list and its sort).
 * The graph is validated (TAURUS_E_INVALID).  Returns after the work
 * completed.
 */
int taurus_reorder_rcm(const taurus_graph* g, int32_t* new_of_old, void* stream);

/*
 * Topology-aware reordering (Sec. 3.8, Alg. 1).  The real positions start
 * from the bootstrap order, r(v) = pi0(v) (pi0: device int32[n], the new ID
 * of each vertex, a permutation of [0, n); NULL = the identity), and each of
 * up to `iterations` (>= 1) updates applies the two minimisers of the
 * dispersion J (Sec. 3.8) to the current positions,
 *     mu(v) = (1/d(v)) sum_{u in N(v)} r(u)
 *     r(w)  = sum_{v : w in N(v)} mu(v)/d(v) / sum_{v : w in N(v)} 1/d(v)
 * with N(v) = v's in-neighbours plus v itself (the self message) and
 * d(v) = |N(v)|, then ranks them, pi = ArgSort(r) with ties by the lower ID.
 * The positions carry over to the next update; the loop ends once an update
 * leaves pi unchanged (pi has converged).
 * Sums are fp64 in a fixed order of the library's own (the same on every
 * run); they agree with a sequential sum within fp64 rounding, so an order
 * can differ from one only between positions that close.
 * Outputs:
 *   new_of_old  device int32[n], written: the order after the last update;
 *   positions   device double[n] or NULL: r after the last update made;
 *   spans       host int64[iterations + 1] or NULL: the total span
 *               C(pi) = sum_v (max - min rank over N(v)) of the bootstrap,
 *               then of the order after each update made;
 *   disp        host double[iterations + 1] or NULL: J of the same orders,
 *               each order's ranks taken as positions with their optimal
 *               centres, sum_v 1/d(v) sum_{u in N(v)} (rank(u) - mean)^2;
 *   *updates    host, may be NULL: updates made.
 * The caller owns every buffer.  Entries of spans and disp past the last
 * update made are left as they were.
 * Errors: TAURUS_E_INVALID for a graph that is not a valid CSR, a pi0 that is
 * not a permutation, or iterations < 1.  Returns after the work completed.
 */
int taurus_reorder_ta(const taurus_graph* g, const int32_t* pi0, int32_t iterations, int32_t* new_of_old,
                      double* positions, int64_t* spans, double* disp, int32_t* updates, void* stream);

/*
 * CSR of the relabelled graph: edge (u, v) becomes (new_of_old[u],
 * new_of_old[v]).  row_off int64[n+1] and col_dst int32[e] are caller-owned
 * device memory, written in canonical form (as taurus_build_csr).
 * new_of_old must be a permutation of [0, n) (else TAURUS_E_INVALID).
 * Returns after the work completed.
 */
int taurus_relabel_graph(const taurus_graph* g, const int32_t* new_of_old, int64_t* row_off, int32_t* col_dst,
                         void* stream);

/*
 * Move rows of row_bytes bytes (a multiple of 4) between vertex numberings:
 * inverse = 0: out[new_of_old[v]] = in[v] (features into the new order);
 * inverse = 1: out[v] = in[new_of_old[v]] (outputs back to the old order).
 * in, out: device [n][row_bytes], not overlapping.  new_of_old must be a
 * permutation (checked; TAURUS_E_INVALID).  Returns after the check; the
 * copy itself is asynchronous on `stream`.
 */
int taurus_permute_rows(const void* in, void* out, int64_t n, int64_t row_bytes, const int32_t* new_of_old,
                        int32_t inverse, void* stream);

/*
 * A plan holds the per-graph structures that layers over one graph and chunk
 * size share: the exact chunk index (every in-edge grouped by source chunk
 * and destination, with each vertex's message count |N-(v)|; Sec. 3.3-3.4:
 * the reader streams contiguous vertex ranges and the orchestrator keeps
 * O(|V|) pending counts) for exact layers, and the in-edges grouped by
 * destination for the fanout sampler of sampled layers.  Each structure is
 * built by the first layer that needs it (on that layer's stream; the graph
 * is validated then: row_off monotone from 0 to e, col_dst in [0, n), rows
 * strictly ascending, no self loops, else TAURUS_E_INVALID) and reused by
 * later layers.  Creating the plan only records the graph and chunk size
 * (stream is unused).  The graph arrays must stay valid and unchanged while
 * the plan or any layer using it lives.  The plan's device memory is held
 * until the plan and every layer that uses it are destroyed.  Layers that
 * share a plan may run on different streams; the first use of a structure
 * must not race with another layer's first use of it from another thread
 * (the plan serialises the build itself).
 */
int taurus_plan_create(const taurus_graph* g, int64_t chunk, void* stream, taurus_plan** out);

/* Release a plan (layers still using it keep its structures alive).  NULL is ignored. */
void taurus_plan_destroy(taurus_plan* plan);

/*
 * Create the state of one layer (Sec. 3.4: one pending-message count per
 * vertex, O(|V|) state; Sec. 3.9 for the sampled message set M(v)): copies
 * the weights, computes degrees and normalisers, draws the fanout sample
 * (fanout > 0), builds or takes the per-chunk destination index, and sets
 * every vertex's pending-message count to |M(v)| + 1 (the self message
 * counts as one arrival).  Without a budget the dense accumulators are
 * allocated first and hold the index build's temporaries until the first
 * push.  *out receives the handle.  Blocks until the index is built.
 * Errors: TAURUS_E_INVALID for bad arguments or a graph that is not a valid
 * simple CSR; TAURUS_E_BUDGET when the budget cannot hold the layer;
 * TAURUS_E_OOM / TAURUS_E_DEVICE from the runtime.  On error *out is NULL.
 */
int taurus_layer_init(const taurus_graph* g, const taurus_layer_desc* d, taurus_layer** out);

/*
 * Stream one source chunk through the layer (Sec. 3.1 broadcast along
 * out-edges; Secs. 3.3-3.6): transform the chunk's rows, push their messages
 * to the destinations and finalise every destination whose last message
 * arrives.  [src_begin, src_end) must be a whole chunk: src_begin = j*chunk,
 * src_end = min(src_begin + chunk, n), because the destination index (which
 * destinations a chunk's sources reach, grouped into work units) is built
 * per chunk at init; other ranges return TAURUS_E_INVALID.
 * x points at the chunk's rows (row src_begin first), row-major
 * [src_end - src_begin][d_in] of in_dtype: device memory if x_on_host = 0,
 * pinned host memory if x_on_host = 1 (copied on the layer's own copy
 * stream into a device staging buffer, overlapping the previous chunk's
 * compute; Sec. 3.3).  x must stay valid and unchanged until the next call
 * on this handle returns.  Chunks may be pushed in any order;
 * each exactly once (a repeat returns TAURUS_E_STATE).  Asynchronous on the
 * layer's stream.
 */
int taurus_push_chunk(taurus_layer* L, int64_t src_begin, int64_t src_end, const void* x,
                      int32_t x_on_host);

/*
 * Wait for the layer's work, check that every destination completed (Sec.
 * 3.6: a vertex graduates once its pending count reaches zero, its output
 * row written by the flush that completes it) and fill *stats (may be
 * NULL).  Returns TAURUS_E_INCOMPLETE (with the count in
 * stats->pending_left) if some destination still has pending messages, e.g.
 * because a chunk was never pushed.  After TAURUS_OK every row of desc.out
 * holds its final value.
 */
int taurus_finalize(taurus_layer* L, taurus_stats* stats);

/*
 * Copy the layer's propagated-edge mask to host memory (Sec. 3.9: the
 * incoming edges the fanout sample keeps): bit i of mask_bits_host[i / 64]
 * (least significant bit first) is set if CSR edge i propagates in this
 * layer (all ones for exact layers).  mask_bits_host has ceil(e/64) words;
 * *n_kept receives the number of set bits (may be NULL).  A sampled layer
 * draws the CSR-order mask on the first call (the same selection as the
 * layer's index), which takes ceil(e/64) words of device memory until
 * destroy.  Synchronises the layer's stream.
 */
int taurus_sampled_edges(taurus_layer* L, uint64_t* mask_bits_host, int64_t* n_kept);

/*
 * Reloads per vertex of a budgeted layer (the distribution the paper's
 * eviction study plots, Sec. 4): counts (host int64[bins], bins >= 2)
 * receives, for i < bins - 1, the number of vertices reloaded exactly i
 * times, and in counts[bins - 1] those reloaded bins - 1 times or more.  An
 * in-core layer reports counts[0] = n.  Any time after init; synchronises
 * the layer's stream.
 */
int taurus_layer_reload_histogram(taurus_layer* L, int64_t* counts, int32_t bins);

/*
 * Chunk loader (Sec. 3.3, Graph Reader: a dedicated reader keeps chunks
 * coming while earlier ones copy and compute; Sec. 3.6, copies overlap
 * compute on separate streams).  The loader fills chunks on host threads,
 * each into one buffer of a ring of pinned host buffers, while the calling
 * thread pushes them in ascending order (taurus_push_chunk with
 * x_on_host = 1: copy on the layer's copy stream, then the chunk's work),
 * so generation or reading, the host-to-device copy and the compute of
 * different chunks overlap.
 *
 * fill(ctx, begin, end, dst) writes rows [begin, end) of the layer's input,
 * row-major [end - begin][d_in] of desc.in_dtype, into dst (pinned host
 * memory owned by the loader) and returns 0, or nonzero to stop the layer.
 * It is called from `threads` loader threads at once (1 .. 64), for
 * different chunks, and must be safe for that.  `ring` pinned buffers of
 * one chunk each (threads + 1 .. 256; 0 picks 2 * threads) hold chunks
 * being filled, filled and waiting, or copying; the ring comes from the
 * library's cache of pinned host buffers (taurus_release_cached_memory)
 * and goes back to it before return.
 *
 * Pushes every chunk of the layer; no chunk may have been pushed before
 * (TAURUS_E_STATE).  Returns when the last chunk is queued and every copy
 * out of the ring is done (the layer's work may still run; call
 * taurus_finalize).  stats (may be NULL) receives the loader's times.
 * Errors: TAURUS_E_INVALID for bad arguments or a fill that returned
 * nonzero (the message names the chunk and the value; the handle is then
 * poisoned, as are push errors after work started); TAURUS_E_OOM when the
 * ring cannot be allocated.
 */
typedef int (*taurus_fill_fn)(void* ctx, int64_t begin, int64_t end, void* dst);

typedef struct {
    int64_t chunks;          /* chunks filled and pushed                          */
    int64_t bytes;           /* host bytes filled (= bytes copied to the device)  */
    double fill_seconds;     /* time inside fill, summed over the loader threads  */
    double wait_seconds;     /* the pushing thread waiting for a filled chunk     */
    double push_seconds;     /* the pushing thread inside taurus_push_chunk       */
    double wall_seconds;     /* the whole call                                    */
} taurus_stream_stats;

int taurus_stream_layer(taurus_layer* L, taurus_fill_fn fill, void* ctx, int32_t threads, int32_t ring,
                        taurus_stream_stats* stats);

/* Release everything the layer allocated.  NULL is ignored. */
void taurus_layer_destroy(taurus_layer* L);

#ifdef __cplusplus
}
#endif

#endif /* TAURUS_H */
