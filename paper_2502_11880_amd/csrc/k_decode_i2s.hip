// Decode GEMV for the I2_S layout (M <= 16 tokens): ternary x int8 accumulation (Eq. 1) on int8 MFMA,
// with the dequantisation epilogue fused.
//
// Weights are HBM-bound: each packed byte is read exactly once, with 16-byte non-temporal loads, one
// contiguous KiB per wave per 256-k block.  A 32-bit word of lane (r, q) holds 16 codes c = t + 1 of
// row r; shifting by 2f and masking 0x03030303 gives the four int8 codes of k = 4f .. 4f+3, which is
// exactly the byte order of the matching activation word.  So the unpacked word feeds the B operand of
// v_mfma_i32_16x16x64_i8 directly (B column = weight row, A row = token; tokens beyond M are zero).
// The codes carry a +1 offset; a second MFMA against an all-ones B gives sum_k xq[m, k] over the same
// k, which is subtracted (exact integers).
//
// Work split: one work group per 16-row group, holding the whole K.  Its 4, 8 or 16 waves take every
// WAVES-th 256-k block, issue all their weight loads up front (a GEMV of a few MB is latency-bound: one
// DRAM round trip should cover it) and reduce through LDS; wave 0 applies the epilogue.  No work group
// depends on another, so no device-wide fence is needed (an agent-scope release writes back the whole
// L2 of the XCD, which costs more than these GEMVs).
#include "bitnet_internal.hpp"

// Tuning constants: 256-k blocks loaded per wave per batch, and the widest work group (in waves).
#ifndef BITNET_DECODE_U
#define BITNET_DECODE_U 2
#endif
#ifndef BITNET_DECODE_MAX_WAVES
#define BITNET_DECODE_MAX_WAVES 16
#endif

namespace bitnet {
namespace {

__device__ __forceinline__ v4i unpack_codes(uint32_t w) {
    v4i b;
    b.x = (int)(w & 0x03030303u);
    b.y = (int)((w >> 2) & 0x03030303u);
    b.z = (int)((w >> 4) & 0x03030303u);
    b.w = (int)((w >> 6) & 0x03030303u);
    return b;
}

__device__ __forceinline__ v4i mfma16x16x64(v4i a, v4i b, v4i c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ v4u load_stream16(const uint8_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p));
}

__device__ __forceinline__ uint32_t word_of(const v4u& v, int j) {
    return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
}

template <int WAVES, int U>
__global__ __launch_bounds__(64 * WAVES) void i2s_decode_kernel(
    const uint8_t* __restrict__ packed, const float* __restrict__ w_scale, const int8_t* __restrict__ xq,
    const float* __restrict__ x_scale, int M, int N, int K, float* __restrict__ y, int32_t* __restrict__ acc_out) {
    __shared__ v4i red[WAVES][64];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int rg = xcd_logical_id(blockIdx.x, gridDim.x);
    const int nkb = (K + kI2sBlockK - 1) / kI2sBlockK;
    const int nfull = K / kI2sBlockK;
    const int q = lane >> 4, r = lane & 15;
    const bool a_on = r < M;                        // A operand: row = token r, 16 k per lane group q
    const int8_t* arow = xq + (size_t)(a_on ? r : 0) * K + 16 * q;
    const uint8_t* wbase = packed + (size_t)rg * 4 * K;
    const v4i ones = {0x01010101, 0x01010101, 0x01010101, 0x01010101};
    const v4i zero = {0, 0, 0, 0};

    v4i acc = zero, rowsum = zero;
    for (int kb = wave; kb < nfull; kb += WAVES * U) {
        v4u wv[U];
        v4i av[U][4];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kbu = kb + WAVES * u;
            if (kbu < nfull) {
                wv[u] = load_stream16(wbase + (size_t)kbu * 1024 + 16 * lane);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    av[u][j] = a_on ? *reinterpret_cast<const v4i*>(arow + kbu * kI2sBlockK + kSubK * j) : zero;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (kb + WAVES * u < nfull) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    acc = mfma16x16x64(av[u][j], unpack_codes(word_of(wv[u], j)), acc);
                    rowsum = mfma16x16x64(av[u][j], ones, rowsum);
                }
            }
        }
    }
    // A short last block (K % 256 != 0): T sub-tiles, lane words 4*T bytes apart.
    if (nfull < nkb && (nfull % WAVES) == wave) {
        const int T = (K - nfull * kI2sBlockK) / kSubK;
        for (int j = 0; j < T; ++j) {
            const v4i a = a_on ? *reinterpret_cast<const v4i*>(arow + nfull * kI2sBlockK + kSubK * j) : zero;
            const uint32_t w = *reinterpret_cast<const uint32_t*>(wbase + (size_t)nfull * 1024 + 4 * T * lane + 4 * j);
            acc = mfma16x16x64(a, unpack_codes(w), acc);
            rowsum = mfma16x16x64(a, ones, rowsum);
        }
    }

    red[wave][lane] = acc - rowsum;
    __syncthreads();
    if (wave != 0) return;
    acc = red[0][lane];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) acc += red[w][lane];

    // Output element v of lane l is D[row 4*(l/16) + v][col l%16]: token m = 4q + v, weight row r.
    const float beta = *w_scale;
    const int n = rg * kRowsPerGroup + r;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int m = 4 * q + v;
        if (m < M) {
            const float sc = beta / x_scale[m];
            y[(size_t)m * N + n] = (float)acc[v] * sc;
            if (acc_out) acc_out[(size_t)m * N + n] = acc[v];
        }
    }
}

}  // namespace

int i2s_decode_waves(int64_t K) {
    const int nkb = (int)((K + kI2sBlockK - 1) / kI2sBlockK);
    const int w = nkb <= 4 ? 4 : nkb <= 8 ? 8 : 16;
    return w < BITNET_DECODE_MAX_WAVES ? w : BITNET_DECODE_MAX_WAVES;
}

hipError_t launch_i2s_decode(const void* packed, const float* w_scale, const int8_t* xq, const float* x_scale,
                             int M, int N, int K, float* y, int32_t* acc, hipStream_t stream) {
    const unsigned grid = (unsigned)(N / kRowsPerGroup);
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    switch (i2s_decode_waves(K)) {
        case 4:
            hipLaunchKernelGGL((i2s_decode_kernel<4, BITNET_DECODE_U>), dim3(grid), dim3(256), 0, stream, pk, w_scale, xq, x_scale,
                               M, N, K, y, acc);
            break;
        case 8:
            hipLaunchKernelGGL((i2s_decode_kernel<8, BITNET_DECODE_U>), dim3(grid), dim3(512), 0, stream, pk, w_scale, xq, x_scale,
                               M, N, K, y, acc);
            break;
        default:
            hipLaunchKernelGGL((i2s_decode_kernel<16, BITNET_DECODE_U>), dim3(grid), dim3(1024), 0, stream, pk, w_scale, xq,
                               x_scale, M, N, K, y, acc);
            break;
    }
    return hipGetLastError();
}

}  // namespace bitnet
