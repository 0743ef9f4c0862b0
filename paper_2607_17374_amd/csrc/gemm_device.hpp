// Device side of the per-chunk transform on the matrix cores: operand
// fragments, the MFMA steps and the row-panel body, shared by the transform
// kernel and the launch that also carries the previous chunk's fix-up.
// Fragment layouts are described at the top of gemm.hip.
#pragma once

#include "device.hpp"
#include "internal.hpp"

namespace taurus {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));

template <int DT>
__device__ inline floatx4 mfma16(uint4 a, uint4 b, floatx4 c) {
    if constexpr (DT == TAURUS_BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                       c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(halfx8, a), __builtin_bit_cast(halfx8, b),
                                                      c, 0, 0, 0);
}

// ---------------------------------------------------- row-panel kernel -----
// A workgroup owns 64 rows and a group of up to NB 16-column blocks (128
// columns for NB = 8); each of its four waves computes 16 rows x all of the
// group's columns, so every X row is read once per column group (once in
// all for widths up to 128).  The group's packed weight fragments are staged
// in LDS one K stage at a time (PIPE_KS k-blocks), and a wave requests all
// of its A fragments of the stage before the matrix-core work.
//   fp32:   k-block = 16 k, fragment = one float4 per lane (4 MFMAs 16x16x4);
//   16-bit: k-block = 32 k, fragment = eight 16-bit values (one 16x16x32 MFMA).
template <int DT>
struct GemmOp;
template <>
struct GemmOp<TAURUS_F32> {
    typedef float4 frag;
    static constexpr int KBLK = 16;
    static __device__ inline floatx4 mma(frag a, frag b, floatx4 c) {
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, c, 0, 0, 0);
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, c, 0, 0, 0);
    }
    static __device__ inline frag load_a(const void* X, int64_t row, int K, int k) {
        return *reinterpret_cast<const float4*>(static_cast<const float*>(X) + row * K + k);
    }
    static __device__ inline frag zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
    // all NB column blocks of one k-block, component-major: consecutive
    // products go to different accumulators instead of one dependent chain
    template <int NB>
    static __device__ inline void mma_all(frag a, const frag (&b)[NB], floatx4 (&acc)[NB]) {
#pragma unroll
        for (int j = 0; j < NB; j++) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b[j].x, acc[j], 0, 0, 0);
#pragma unroll
        for (int j = 0; j < NB; j++) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b[j].y, acc[j], 0, 0, 0);
#pragma unroll
        for (int j = 0; j < NB; j++) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b[j].z, acc[j], 0, 0, 0);
#pragma unroll
        for (int j = 0; j < NB; j++) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b[j].w, acc[j], 0, 0, 0);
    }
};
template <int DT>
struct GemmOp16 {
    typedef uint4 frag;
    static constexpr int KBLK = 32;
    static __device__ inline floatx4 mma(frag a, frag b, floatx4 c) { return mfma16<DT>(a, b, c); }
    static __device__ inline frag load_a(const void* X, int64_t row, int K, int k) {
        return *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(X) + row * K + k);
    }
    static __device__ inline frag zero() { return make_uint4(0, 0, 0, 0); }
    template <int NB>
    static __device__ inline void mma_all(frag a, const frag (&b)[NB], floatx4 (&acc)[NB]) {
#pragma unroll
        for (int j = 0; j < NB; j++) acc[j] = mfma16<DT>(a, b[j], acc[j]);
    }
};
template <>
struct GemmOp<TAURUS_BF16> : GemmOp16<TAURUS_BF16> {};
template <>
struct GemmOp<TAURUS_F16> : GemmOp16<TAURUS_F16> {};

constexpr int PANEL_ROWS = 64;

// Whether a transform writes Y with streaming stores: rows of whole 128-byte
// lines (a row stride that is a multiple of 32 floats) and a Y of more than
// 64 MB, twice the L2 of the chip's eight XCDs, which its scatter would not
// find in L2 anyway.  Measured: the 1M-vertex GCN's 33.5 MB Y scattered 4%
// slower when streamed; the 100M-vertex GraphSAGE's 92 to 134 MB chunks
// transform 7% faster with no change in the scatter.
inline bool transform_streams(int64_t M, int Nc) { return Nc % 32 == 0 && M * (int64_t)Nc * 4 > ((int64_t)64 << 20); }

// The weights go through two LDS buffers of PIPE_KS k-blocks each: while a
// stage's products run, the next stage's weight fragments (into registers,
// then into the other buffer) and A fragments are already in flight, so
// the workgroups' loads overlap their matrix-core work (all of a chunk's
// workgroups are resident at once and would otherwise load and multiply in
// lockstep).  One barrier per stage.  PANEL_NB: 16-column blocks per
// workgroup (8 = 128 columns; 4 for narrow outputs).  Run by a whole
// workgroup of 256 threads for the panel (bx, by): rows [64 bx, 64 bx + 64),
// column blocks [PANEL_NB by, PANEL_NB by + PANEL_NB).  sB is the calling
// kernel's own LDS array of PanelLds<DT, PANEL_NB> (an array declared here
// would be one LDS variable shared by every kernel of the file, which the
// compiler then addresses less directly).
constexpr int PIPE_KS = 2;
template <int DT, int PANEL_NB>
struct PanelLds {
    static constexpr int SF = PIPE_KS * PANEL_NB * 64;  // fragments per stage
    typename GemmOp<DT>::frag b[2][SF];
};
// The body with the row mapping and the epilogue as parameters: logical row
// r of the panel reads row arow(r) of X; for each row r < M the epilogue's
// row(r) returns a per-row writer w, and w(col, value) stores each product
// of that row, column col < Nc.
template <int DT, int PANEL_NB, class ARow>
__device__ __attribute__((always_inline)) inline void gemm_panel_compute(const void* __restrict__ X, int64_t M,
                                        int K, const typename GemmOp<DT>::frag* __restrict__ Wp, int NBP, int bx,
                                        int by, PanelLds<DT, PANEL_NB>& lds, ARow arow,
                                        floatx4 (&acc)[PANEL_NB]) {
    typedef GemmOp<DT> Op;
    typedef typename Op::frag frag;
    constexpr int SF = PanelLds<DT, PANEL_NB>::SF;
    constexpr int PER = SF / 256;                // of which each thread stages
    static_assert(SF % 256 == 0, "whole fragments per thread");
    auto& sB = lds.b;
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int li = lane & 15, lk = lane >> 4;
    const int nb0 = by * PANEL_NB;
    const int nbs = min(PANEL_NB, NBP - nb0);
    const int64_t row = (int64_t)bx * PANEL_ROWS + wave * 16 + li;
    const int KB = (K + Op::KBLK - 1) / Op::KBLK;
    const int nst = (KB + PIPE_KS - 1) / PIPE_KS;
    auto load_w = [&](int st, frag (&r)[PER]) {
#pragma unroll
        for (int q = 0; q < PER; q++) {
            const int i = q * 256 + tid;
            const int kk = i / (PANEL_NB * 64), rr = i - kk * (PANEL_NB * 64), j = rr >> 6, l = rr & 63;
            const int kb = st * PIPE_KS + kk;
            r[q] = (kb < KB && j < nbs) ? Wp[((int64_t)kb * NBP + nb0 + j) * 64 + l] : Op::zero();
        }
    };
    auto load_a = [&](int st, frag (&a)[PIPE_KS]) {
#pragma unroll
        for (int kk = 0; kk < PIPE_KS; kk++) {
            const int kb = st * PIPE_KS + kk;
            const int k = kb * Op::KBLK + (Op::KBLK / 4) * lk;
            a[kk] = (kb < KB && row < M && k < K) ? Op::load_a(X, arow(row), K, k) : Op::zero();
        }
    };
#pragma unroll
    for (int j = 0; j < PANEL_NB; j++) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    frag rw[PER], a[PIPE_KS];
    load_w(0, rw);
    load_a(0, a);
#pragma unroll
    for (int q = 0; q < PER; q++) sB[0][q * 256 + tid] = rw[q];
    __syncthreads();
    for (int st = 0; st < nst; st++) {
        const bool more = st + 1 < nst;
        frag an[PIPE_KS];
        if (more) {
            load_w(st + 1, rw);
            load_a(st + 1, an);
        }
#pragma unroll
        for (int kk = 0; kk < PIPE_KS; kk++) {
            frag b[PANEL_NB];
#pragma unroll
            for (int j = 0; j < PANEL_NB; j++) b[j] = sB[st & 1][(kk * PANEL_NB + j) * 64 + lane];
            Op::template mma_all<PANEL_NB>(a[kk], b, acc);
        }
        if (more) {
            // the other buffer was last read in the previous stage, before its barrier
#pragma unroll
            for (int q = 0; q < PER; q++) sB[(st + 1) & 1][q * 256 + tid] = rw[q];
#pragma unroll
            for (int kk = 0; kk < PIPE_KS; kk++) a[kk] = an[kk];
        }
        __syncthreads();
    }
}

// The panel with a per-element epilogue: lane (li, lk) of wave w holds rows
// 64 bx + 16 w + 4 lk + r (r = 0..3) of column 16 (PANEL_NB by + j) + li in
// acc[j][r].
template <int DT, int PANEL_NB, class ARow, class Epi>
__device__ __attribute__((always_inline)) inline void gemm_panel_core(const void* __restrict__ X, int64_t M, int K,
                                        const typename GemmOp<DT>::frag* __restrict__ Wp, int NBP, int Nc, int bx,
                                        int by, PanelLds<DT, PANEL_NB>& lds, ARow arow, Epi epi) {
    floatx4 acc[PANEL_NB];
    gemm_panel_compute<DT, PANEL_NB>(X, M, K, Wp, NBP, bx, by, lds, arow, acc);
    const int lane = threadIdx.x & 63, li = lane & 15, lk = lane >> 4;
    const int nb0 = by * PANEL_NB, nbs = min(PANEL_NB, NBP - nb0);
    const int64_t rbase = (int64_t)bx * PANEL_ROWS + (threadIdx.x >> 6) * 16 + 4 * lk;
#pragma unroll
    for (int r = 0; r < 4; r++) {
        const int64_t orow = rbase + r;
        if (orow >= M) continue;
        auto w = epi.row(orow);
#pragma unroll
        for (int j = 0; j < PANEL_NB; j++) {
            const int col = (nb0 + j) * 16 + li;
            if (j < nbs && col < Nc) w(col, acc[j][r]);
        }
    }
}

// GraphSAGE self messages taken by the chunk's transform (in-core layers).
// Vertex v = first_row + r of the chunk whose self message is not a slot of
// a segment from its own chunk (no OWN_SEGMENT) receives W_self h_v straight
// from the products of its self-half columns [self_col, self_col + d_o),
// with weight 1 as in a flush: added to its accumulator row (or written as
// the row when nothing has arrived yet), or, when it is v's last arrival,
// finalised into its output row as act(acc + b).  Y then holds only the
// aggregation half of such rows.  The counts are only read here (a row's
// columns are split over several workgroups): the scatter that follows
// takes the self arrival off.  own == nullptr: every row goes to Y.
struct SelfFlush {
    const uint8_t* own;   // per vertex: chunk-index flags
    const int2* cnt;      // per vertex: {pending, expected}
    float* acc;           // [n][d_o] fp32 accumulator rows
    void* out;            // [n][d_o] output rows in out_dtype
    const float* bias;    // [d_o]
    int64_t first_row;    // first vertex of the chunk
    int self_col, d_o, relu, out_dtype;
};

// A column group [c0, c0 + tw) of the products that holds self-half columns.
__device__ inline bool self_group(const SelfFlush& sf, int c0, int tw) {
    return sf.own && c0 < sf.self_col + sf.d_o && c0 + tw > sf.self_col;
}

// What a panel's self messages need to know of its 64 rows, one bit per row
// (the same in every wave of the workgroup): the row's self message is taken
// here (no OWN_SEGMENT), nothing has been accumulated for it yet, and it is
// the row's last arrival.
struct SelfRows {
    uint64_t take, fresh, last;
};

// The products of one panel leave through LDS (the weight buffers are free
// once the last stage is done): a 64 x 16 PANEL_NB fp32 tile, written in
// the matrix cores' layout and read back row-major, so that each wave
// stores whole 16-byte pieces of consecutive columns (two full 512-byte
// rows per store for 128 columns) instead of 64-byte pieces of four rows.
// Columns are XOR-swizzled by 16 with bit 2 of the row, so the four row
// groups of a store into the tile fall on distinct bank halves.  Rows are
// scaled by rscale when given.  stream: write with streaming (non-temporal)
// stores, for a Y too large to stay in L2 until its scatter reads it.
// Ends with the tile read: a caller that writes the buffers again first
// passes a barrier.
template <int DT, int PANEL_NB>
__device__ __attribute__((always_inline)) inline void store_panel_staged(const floatx4 (&acc)[PANEL_NB],
                                        PanelLds<DT, PANEL_NB>& lds, int64_t M, int Nc,
                                        const float* __restrict__ rscale, float* __restrict__ Y, int bx, int by,
                                        bool stream, const SelfFlush& sf, const SelfRows& sr) {
    constexpr int TW = PANEL_NB * 16;  // tile width (fp32 columns)
    static_assert(sizeof(lds.b) >= (size_t)PANEL_ROWS * TW * 4, "the weight buffers hold the output tile");
    float* tile = reinterpret_cast<float*>(&lds.b[0][0]);
    const int tid = threadIdx.x, lane = tid & 63, li = lane & 15, lk = lane >> 4;
    const int c0 = by * TW;  // first column of the group
    constexpr int Q = TW / 4;  // float4 per tile row
    constexpr int IT = PANEL_ROWS * Q / 256;  // float4 per thread
    // Thread tid stores float4 i of the tile at row (256 i + tid) / Q, column
    // 4 ((256 i + tid) % Q) of the group.  A group with self-half columns
    // (GraphSAGE: rows are not scaled) requests the accumulator pieces its
    // self messages need before the tile goes through LDS, so that their
    // loads overlap the staging.
    const bool selfs = self_group(sf, c0, TW);
    auto takes = [&](int row, int col) {
        return col >= sf.self_col && col < sf.self_col + sf.d_o && ((sr.take >> row) & 1);
    };
    float4 prev[IT];
    if (selfs) {
#pragma unroll
        for (int i = 0; i < IT; i++) {
            const int q = i * 256 + tid, row = q / Q, c = (q % Q) * 4;
            const int64_t grow = (int64_t)bx * PANEL_ROWS + row;
            const int col = c0 + c;
            prev[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (grow < M && col < Nc && takes(row, col) && !((sr.fresh >> row) & 1))
                prev[i] = *reinterpret_cast<const float4*>(sf.acc + (sf.first_row + grow) * sf.d_o + (col - sf.self_col));
        }
    }
#pragma unroll
    for (int r = 0; r < 4; r++) {
        const int row = (tid >> 6) * 16 + 4 * lk + r;
        const int sw = ((row >> 2) & 1) << 4;
#pragma unroll
        for (int j = 0; j < PANEL_NB; j++) tile[row * TW + ((j * 16 + li) ^ sw)] = acc[j][r];
    }
    __syncthreads();
    auto put = [&](float* dst, float4 v) {
        if (stream)
            __builtin_nontemporal_store(floatx4{v.x, v.y, v.z, v.w}, reinterpret_cast<floatx4*>(dst));
        else
            *reinterpret_cast<float4*>(dst) = v;
    };
#pragma unroll
    for (int i = 0; i < IT; i++) {
        const int q = i * 256 + tid, row = q / Q, c = (q % Q) * 4;
        const int64_t grow = (int64_t)bx * PANEL_ROWS + row;
        const int col = c0 + c;
        if (grow >= M || col >= Nc) continue;
        const int sw = ((row >> 2) & 1) << 4;
        float4 x = *reinterpret_cast<const float4*>(tile + row * TW + (c ^ sw));
        if (!selfs || !takes(row, col)) {
            if (rscale) {
                const float sc = rscale[grow];
                x.x *= sc;
                x.y *= sc;
                x.z *= sc;
                x.w *= sc;
            }
            put(Y + grow * Nc + col, x);
            continue;
        }
        // v's self message: add, or finalise on its last arrival
        const int64_t v = sf.first_row + grow;
        const int ac = col - sf.self_col;
        const float4 t = make_float4(x.x + prev[i].x, x.y + prev[i].y, x.z + prev[i].z, x.w + prev[i].w);
        if ((sr.last >> row) & 1) {
            const float4 b = *reinterpret_cast<const float4*>(sf.bias + ac);
            float4 z = make_float4(t.x + b.x, t.y + b.y, t.z + b.z, t.w + b.w);
            if (sf.relu) {
                z.x = fmaxf(z.x, 0.f); z.y = fmaxf(z.y, 0.f);
                z.z = fmaxf(z.z, 0.f); z.w = fmaxf(z.w, 0.f);
            }
            store_out4(sf.out, sf.out_dtype, v * sf.d_o + ac, z);
        } else {
            put(sf.acc + v * sf.d_o + ac, t);
        }
    }
}

// Y = X W, rows [64 bx, 64 bx + 64) and column blocks [PANEL_NB by,
// PANEL_NB by + PANEL_NB), through the staged store (with the self
// messages sf takes).
template <int DT, int PANEL_NB>
__device__ __attribute__((always_inline)) inline void gemm_panel_block(const void* __restrict__ X, int64_t M, int K,
                                        const typename GemmOp<DT>::frag* __restrict__ Wp, int NBP, int Nc,
                                        const float* __restrict__ rscale, float* __restrict__ Y, int bx, int by,
                                        PanelLds<DT, PANEL_NB>& lds, bool stream, const SelfFlush& sf) {
    // a group with self messages: lane l of every wave reads row l's flag
    // and counts, and the wave turns them into SelfRows (uniform, so they
    // hold no vector registers through the products); the epilogue then
    // waits on the accumulator rows alone
    SelfRows sr{0, 0, 0};
    if (self_group(sf, by * PANEL_NB * 16, PANEL_NB * 16)) {
        const int64_t r = (int64_t)bx * PANEL_ROWS + (threadIdx.x & 63);
        uint32_t fl = OWN_SEGMENT;
        int2 pe = make_int2(0, 0);
        if (r < M) {
            fl = sf.own[sf.first_row + r];
            pe = sf.cnt[sf.first_row + r];
        }
        sr.take = __ballot(!(fl & OWN_SEGMENT));
        sr.fresh = __ballot(pe.x == pe.y);
        sr.last = __ballot(pe.x == 1);
    }
    floatx4 acc[PANEL_NB];
    gemm_panel_compute<DT, PANEL_NB>(X, M, K, Wp, NBP, bx, by, lds, [](int64_t r) { return r; }, acc);
    // every wave is past the last stage's barrier: the buffers are free
    store_panel_staged<DT, PANEL_NB>(acc, lds, M, Nc, rscale, Y, bx, by, stream, sf, sr);
}

}  // namespace taurus
