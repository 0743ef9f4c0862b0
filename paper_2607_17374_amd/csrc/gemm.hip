// Per-chunk feature transform Y = X_c . W on the matrix cores.
//
// Transforming a source's row before it is broadcast is exact by linearity:
// the paper uses the same identity for its GraphSAGE weight split (Sec. 3.9,
// W [h_agg || h_v] = W_agg h_agg + W_self h_v), and the same holds for the
// normalised sums of GCN and the means of GraphSAGE because the aggregate
// is linear in the messages.
//
// fp32 inputs use v_mfma_f32_16x16x4_f32.  Operand fragments for a 16-wide
// K step are read as one float4 per lane: lane l holds
//     A: X[row0 + l%16][k0 + 4*(l/16) + c],   c = 0..3
//     B: W[k0 + 4*(l/16) + c][col0 + l%16]
// and four MFMAs (one per c) consume them.  Each MFMA contracts over the
// lane-group index l/16; across the four of them every k in [k0, k0+16) is
// used exactly once, so the permuted K order does not change the product.
// The weights are repacked once per layer so that each lane's B float4 is
// contiguous (a 1 KiB coalesced load per wave and K step).
//
// bf16 and fp16 inputs use v_mfma_f32_16x16x32_{bf16,f16} with fp32
// accumulation: lane l holds eight consecutive k of row (col) l%16 starting
// at k0 + 8*(l/16).  A and B use the same lane/element-to-k assignment, so
// each MFMA again contracts every k of its 32-wide step exactly once.
#include <cstring>

#include "gemm_device.hpp"

namespace taurus {


// packed weights cover whole 64-column groups (zero padded)
int gemm_packed_blocks_n(int nc) { return (int)ceil_div(nc, 64) * 4; }
int gemm_packed_blocks_k(int k) { return (int)ceil_div(k, 16); }

// Host-side repack of a row-major [K][Nc] fp32 matrix into MFMA B fragments.
void gemm_pack_weights_f32(const float* W, int K, int Nc, std::vector<float>& packed) {
    const int KB = gemm_packed_blocks_k(K), NBP = gemm_packed_blocks_n(Nc);
    packed.assign((size_t)KB * NBP * 64 * 4, 0.0f);
    for (int kb = 0; kb < KB; kb++)
        for (int nb = 0; nb < NBP; nb++)
            for (int l = 0; l < 64; l++)
                for (int c = 0; c < 4; c++) {
                    const int k = kb * 16 + 4 * (l >> 4) + c, col = nb * 16 + (l & 15);
                    float w = (k < K && col < Nc) ? W[(size_t)k * Nc + col] : 0.0f;
                    packed[(((size_t)kb * NBP + nb) * 64 + l) * 4 + c] = w;
                }
}

// ---------------------------------------------------------- 16-bit inputs --

int gemm_packed_blocks_k16(int k) { return (int)ceil_div(k, 32); }

static uint16_t host_f32_to_bf16(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);  // quiet NaN
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}
static uint16_t host_f32_to_f16(float f) {
    const _Float16 h = (_Float16)f;  // round to nearest even
    uint16_t b;
    std::memcpy(&b, &h, 2);
    return b;
}

// Host-side repack of a row-major [K][Nc] fp32 matrix into 16-bit MFMA B
// fragments (values rounded to nearest even in the input type).
void gemm_pack_weights_16(const float* W, int K, int Nc, int dtype, std::vector<uint16_t>& packed) {
    const int KB = gemm_packed_blocks_k16(K), NBP = gemm_packed_blocks_n(Nc);
    packed.assign((size_t)KB * NBP * 64 * 8, 0);
    for (int kb = 0; kb < KB; kb++)
        for (int nb = 0; nb < NBP; nb++)
            for (int l = 0; l < 64; l++)
                for (int c = 0; c < 8; c++) {
                    const int k = kb * 32 + 8 * (l >> 4) + c, col = nb * 16 + (l & 15);
                    const float w = (k < K && col < Nc) ? W[(size_t)k * Nc + col] : 0.0f;
                    packed[(((size_t)kb * NBP + nb) * 64 + l) * 8 + c] =
                        dtype == TAURUS_BF16 ? host_f32_to_bf16(w) : host_f32_to_f16(w);
                }
}

template <int DT, int PANEL_NB>
__global__ __launch_bounds__(256) void k_gemm_panel(const void* __restrict__ X, int64_t M, int K,
                                                    const typename GemmOp<DT>::frag* __restrict__ Wp, int NBP,
                                                    int Nc, const float* __restrict__ rscale,
                                                    float* __restrict__ Y, int stream, SelfFlush sf) {
    __shared__ PanelLds<DT, PANEL_NB> lds;
    // With self messages the column groups start at the first one holding
    // self-half columns: those workgroups wait on accumulator rows, and
    // dispatched first they overlap the purely streaming groups that follow
    // instead of forming the launch's tail.
    const int by = sf.own ? (int)((blockIdx.y + sf.self_col / (PANEL_NB * 16)) % gridDim.y) : (int)blockIdx.y;
    gemm_panel_block<DT, PANEL_NB>(X, M, K, Wp, NBP, Nc, rscale, Y, blockIdx.x, by, lds, stream != 0, sf);
}

template <int DT>
static void launch_panel(const void* X, int64_t M, int K, const void* Wp, int Nc, const float* rscale, float* Y,
                         const SelfFlush* sf, hipStream_t s) {
    const int NBP = gemm_packed_blocks_n(Nc);
    const auto* w = static_cast<const typename GemmOp<DT>::frag*>(Wp);
    const int stream = transform_streams(M, Nc) ? 1 : 0;
    const SelfFlush f = sf ? *sf : SelfFlush{};
    if (f.own && (rscale || f.self_col + f.d_o > Nc || f.self_col % 4 || f.d_o % 4))
        fail(TAURUS_E_INVALID, "self messages in the transform need unscaled rows and a self half inside Y");
    if (NBP <= 4) {
        dim3 grid((unsigned)ceil_div(M, PANEL_ROWS), 1);
        k_gemm_panel<DT, 4><<<grid, 256, 0, s>>>(X, M, K, w, NBP, Nc, rscale, Y, stream, f);
    } else {
        dim3 grid((unsigned)ceil_div(M, PANEL_ROWS), (unsigned)ceil_div(NBP, 8));
        k_gemm_panel<DT, 8><<<grid, 256, 0, s>>>(X, M, K, w, NBP, Nc, rscale, Y, stream, f);
    }
    TAURUS_CHECK_LAUNCH();
}

void gemm_f32(const float* X, int64_t M, int K, const float* Wp, int Nc, const float* rscale, float* Y,
              const SelfFlush* sf, hipStream_t s) {
    if (M <= 0) return;
    launch_panel<TAURUS_F32>(X, M, K, Wp, Nc, rscale, Y, sf, s);
}

void gemm_16(const uint16_t* X, int dtype, int64_t M, int K, const uint16_t* Wp, int Nc, const float* rscale,
             float* Y, const SelfFlush* sf, hipStream_t s) {
    if (M <= 0) return;
    if (dtype == TAURUS_BF16) launch_panel<TAURUS_BF16>(X, M, K, Wp, Nc, rscale, Y, sf, s);
    else launch_panel<TAURUS_F16>(X, M, K, Wp, Nc, rscale, Y, sf, s);
}

}  // namespace taurus
