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

#include "internal.hpp"

namespace taurus {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int GEMM_WM = 2;  // 16-row blocks per wave
constexpr int GEMM_WN = 2;  // 16-col blocks per wave
constexpr int GEMM_TM = 2 * GEMM_WM * 16;  // workgroup tile rows (2 waves along M)
constexpr int GEMM_TN = 2 * GEMM_WN * 16;  // workgroup tile cols (2 waves along N)

int gemm_packed_blocks_n(int nc) { return (int)ceil_div(nc, GEMM_TN) * (GEMM_TN / 16); }
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

__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ X, int64_t M, int K,
                                                  const float4* __restrict__ Wp, int NBP, int Nc,
                                                  const float* __restrict__ rscale, float* __restrict__ Y) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int wm = wave & 1, wn = wave >> 1;
    const int64_t m0 = (int64_t)blockIdx.x * GEMM_TM + wm * (GEMM_WM * 16);
    const int nb0 = blockIdx.y * (GEMM_TN / 16) + wn * GEMM_WN;
    const int li = lane & 15, lk = lane >> 4;
    floatx4 acc[GEMM_WM][GEMM_WN];
#pragma unroll
    for (int i = 0; i < GEMM_WM; i++)
#pragma unroll
        for (int j = 0; j < GEMM_WN; j++) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int KB = (K + 15) >> 4;
    for (int kb = 0; kb < KB; kb++) {
        const int k = kb * 16 + 4 * lk;
        float4 a[GEMM_WM], b[GEMM_WN];
#pragma unroll
        for (int i = 0; i < GEMM_WM; i++) {
            const int64_t row = m0 + i * 16 + li;
            a[i] = (row < M && k < K) ? *reinterpret_cast<const float4*>(X + row * K + k)
                                      : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int j = 0; j < GEMM_WN; j++) b[j] = Wp[((int64_t)kb * NBP + nb0 + j) * 64 + lane];
#pragma unroll
        for (int i = 0; i < GEMM_WM; i++)
#pragma unroll
            for (int j = 0; j < GEMM_WN; j++) {
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].x, b[j].x, acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].y, b[j].y, acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].z, b[j].z, acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].w, b[j].w, acc[i][j], 0, 0, 0);
            }
    }
    // D fragment: lane l holds rows 4*(l/16) + r, column l%16
#pragma unroll
    for (int i = 0; i < GEMM_WM; i++)
#pragma unroll
        for (int r = 0; r < 4; r++) {
            const int64_t row = m0 + i * 16 + 4 * lk + r;
            if (row >= M) continue;
            const float sc = rscale ? rscale[row] : 1.0f;
#pragma unroll
            for (int j = 0; j < GEMM_WN; j++) {
                const int col = (nb0 + j) * 16 + li;
                if (col < Nc) Y[row * Nc + col] = acc[i][j][r] * sc;
            }
        }
}

// ---------------------------------------------------------- 16-bit inputs --
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 halfx8 __attribute__((ext_vector_type(8)));

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

template <int DT>
__device__ inline floatx4 mfma16(uint4 a, uint4 b, floatx4 c) {
    if constexpr (DT == TAURUS_BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                       c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(halfx8, a), __builtin_bit_cast(halfx8, b),
                                                      c, 0, 0, 0);
}

// X is [M][K] 16-bit, K a multiple of 8 (each lane's eight k are one 16-byte load).
template <int DT>
__global__ __launch_bounds__(256) void k_gemm_16(const uint16_t* __restrict__ X, int64_t M, int K,
                                                 const uint4* __restrict__ Wp, int NBP, int Nc,
                                                 const float* __restrict__ rscale, float* __restrict__ Y) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int wm = wave & 1, wn = wave >> 1;
    const int64_t m0 = (int64_t)blockIdx.x * GEMM_TM + wm * (GEMM_WM * 16);
    const int nb0 = blockIdx.y * (GEMM_TN / 16) + wn * GEMM_WN;
    const int li = lane & 15, lk = lane >> 4;
    floatx4 acc[GEMM_WM][GEMM_WN];
#pragma unroll
    for (int i = 0; i < GEMM_WM; i++)
#pragma unroll
        for (int j = 0; j < GEMM_WN; j++) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const int KB = (K + 31) >> 5;
    for (int kb = 0; kb < KB; kb++) {
        const int k = kb * 32 + 8 * lk;
        uint4 a[GEMM_WM], b[GEMM_WN];
#pragma unroll
        for (int i = 0; i < GEMM_WM; i++) {
            const int64_t row = m0 + i * 16 + li;
            a[i] = (row < M && k < K) ? *reinterpret_cast<const uint4*>(X + row * K + k) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < GEMM_WN; j++) b[j] = Wp[((int64_t)kb * NBP + nb0 + j) * 64 + lane];
#pragma unroll
        for (int i = 0; i < GEMM_WM; i++)
#pragma unroll
            for (int j = 0; j < GEMM_WN; j++) acc[i][j] = mfma16<DT>(a[i], b[j], acc[i][j]);
    }
#pragma unroll
    for (int i = 0; i < GEMM_WM; i++)
#pragma unroll
        for (int r = 0; r < 4; r++) {
            const int64_t row = m0 + i * 16 + 4 * lk + r;
            if (row >= M) continue;
            const float sc = rscale ? rscale[row] : 1.0f;
#pragma unroll
            for (int j = 0; j < GEMM_WN; j++) {
                const int col = (nb0 + j) * 16 + li;
                if (col < Nc) Y[row * Nc + col] = acc[i][j][r] * sc;
            }
        }
}

void gemm_16(const uint16_t* X, int dtype, int64_t M, int K, const uint16_t* Wp, int Nc, const float* rscale,
             float* Y, hipStream_t s) {
    if (M <= 0) return;
    const int NBP = gemm_packed_blocks_n(Nc);
    dim3 grid((unsigned)ceil_div(M, GEMM_TM), (unsigned)(NBP / (GEMM_TN / 16)));
    const uint4* wp = reinterpret_cast<const uint4*>(Wp);
    if (dtype == TAURUS_BF16) k_gemm_16<TAURUS_BF16><<<grid, 256, 0, s>>>(X, M, K, wp, NBP, Nc, rscale, Y);
    else k_gemm_16<TAURUS_F16><<<grid, 256, 0, s>>>(X, M, K, wp, NBP, Nc, rscale, Y);
    TAURUS_CHECK_LAUNCH();
}

void gemm_f32(const float* X, int64_t M, int K, const float* Wp, int Nc, const float* rscale, float* Y,
              hipStream_t s) {
    if (M <= 0) return;
    const int NBP = gemm_packed_blocks_n(Nc);
    dim3 grid((unsigned)ceil_div(M, GEMM_TM), (unsigned)(NBP / (GEMM_TN / 16)));
    k_gemm_f32<<<grid, 256, 0, s>>>(X, M, K, reinterpret_cast<const float4*>(Wp), NBP, Nc, rscale, Y);
    TAURUS_CHECK_LAUNCH();
}

}  // namespace taurus
