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
// Work split: a work group (4 waves) owns NT row groups (16*NT rows) and a range of 256-k blocks;
// waves take every 4th block.  Waves reduce through LDS; when K is split over several work groups the
// partial int32 sums go to the workspace and the last group to finish (an atomic ticket per tile) adds
// them in split order and applies the epilogue.  Ticket counters are reset to zero by that group.
#include "bitnet_internal.hpp"

#include <algorithm>

namespace bitnet {
namespace {

constexpr int kWaves = 4;
constexpr int kBlock = 64 * kWaves;

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

template <int NT, int U>
__global__ __launch_bounds__(kBlock) void i2s_decode_kernel(
    const uint8_t* __restrict__ packed, const float* __restrict__ w_scale, const int8_t* __restrict__ xq,
    const float* __restrict__ x_scale, int M, int N, int K, float* __restrict__ y, int32_t* __restrict__ acc_out,
    int32_t* __restrict__ partial, unsigned* __restrict__ tickets, int splits, int kb_per_split) {
    __shared__ v4i red[kWaves][NT][64];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int L = xcd_logical_id(blockIdx.x, gridDim.x);
    const int tile = L / splits, sp = L - tile * splits;
    const int nkb = (K + kI2sBlockK - 1) / kI2sBlockK;
    const int nfull = K / kI2sBlockK;
    const int kb0 = sp * kb_per_split;
    const int kb1 = min(kb0 + kb_per_split, nkb);
    const int q = lane >> 4, r = lane & 15;
    const bool a_on = r < M;                        // A operand: row = token r, 16 k per lane group q
    const int8_t* arow = xq + (size_t)(a_on ? r : 0) * K + 16 * q;
    const size_t rg_bytes = (size_t)4 * K;
    const uint8_t* wbase = packed + (size_t)tile * NT * rg_bytes;
    const v4i ones = {0x01010101, 0x01010101, 0x01010101, 0x01010101};
    const v4i zero = {0, 0, 0, 0};

    v4i acc[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = zero;
    v4i rowsum = zero;

    const int full_end = min(kb1, nfull);
    for (int kb = kb0 + wave; kb < full_end; kb += kWaves * U) {
        v4u wv[U][NT];
        v4i av[U][4];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kbu = kb + kWaves * u;
            if (kbu < full_end) {
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    wv[u][t] = load_stream16(wbase + t * rg_bytes + (size_t)kbu * 1024 + 16 * lane);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    av[u][j] = a_on ? *reinterpret_cast<const v4i*>(arow + kbu * kI2sBlockK + kSubK * j) : zero;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (kb + kWaves * u < full_end) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        const uint32_t w = j == 0 ? wv[u][t].x : j == 1 ? wv[u][t].y : j == 2 ? wv[u][t].z : wv[u][t].w;
                        acc[t] = mfma16x16x64(av[u][j], unpack_codes(w), acc[t]);
                    }
                    rowsum = mfma16x16x64(av[u][j], ones, rowsum);
                }
            }
        }
    }
    // A short last block (K % 256 != 0): T sub-tiles, lane words 4*T bytes apart.
    if (nfull < nkb && nkb - 1 >= kb0 && nkb - 1 < kb1 && ((nkb - 1 - kb0) % kWaves) == wave) {
        const int kbu = nkb - 1;
        const int T = (K - nfull * kI2sBlockK) / kSubK;
        for (int j = 0; j < T; ++j) {
            const v4i a = a_on ? *reinterpret_cast<const v4i*>(arow + kbu * kI2sBlockK + kSubK * j) : zero;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const uint32_t w = *reinterpret_cast<const uint32_t*>(wbase + t * rg_bytes + (size_t)kbu * 1024 +
                                                                      4 * T * lane + 4 * j);
                acc[t] = mfma16x16x64(a, unpack_codes(w), acc[t]);
            }
            rowsum = mfma16x16x64(a, ones, rowsum);
        }
    }

#pragma unroll
    for (int t = 0; t < NT; ++t) {
        acc[t] -= rowsum;
        red[wave][t][lane] = acc[t];
    }
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = red[0][t][lane] + red[1][t][lane] + red[2][t][lane] + red[3][t][lane];

    // Output element v of lane l is D[row 4*(l/16) + v][col l%16]: token m = 4q + v, weight row r.
    if (splits > 1) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int n = (tile * NT + t) * kRowsPerGroup + r;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = 4 * q + v;
                if (m < M)
                    __hip_atomic_store(partial + ((size_t)sp * M + m) * N + n, acc[t][v], __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        __threadfence();
        unsigned prev = 0u;
        if (lane == 0) prev = atomicAdd(tickets + tile, 1u);
        prev = __shfl(prev, 0, 64);
        if (prev != (unsigned)(splits - 1)) return;
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int n = (tile * NT + t) * kRowsPerGroup + r;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = 4 * q + v;
                int s = 0;
                if (m < M)
                    for (int p = 0; p < splits; ++p)
                        s += __hip_atomic_load(partial + ((size_t)p * M + m) * N + n, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                acc[t][v] = s;
            }
        }
        if (lane == 0) tickets[tile] = 0u;
    }

    const float beta = *w_scale;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int n = (tile * NT + t) * kRowsPerGroup + r;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int m = 4 * q + v;
            if (m < M) {
                const float sc = beta / x_scale[m];
                y[(size_t)m * N + n] = (float)acc[t][v] * sc;
                if (acc_out) acc_out[(size_t)m * N + n] = acc[t][v];
            }
        }
    }
}

template <int NT>
hipError_t launch_nt(const DecodePlan& p, const void* packed, const float* w_scale, const int8_t* xq,
                     const float* x_scale, int M, int N, int K, float* y, int32_t* acc, void* ws,
                     hipStream_t stream) {
    int32_t* partial = static_cast<int32_t*>(ws);
    unsigned* tickets = reinterpret_cast<unsigned*>(static_cast<uint8_t*>(ws) +
                                                    (size_t)p.splits * 16 * N * sizeof(int32_t));
    const unsigned grid = (unsigned)(p.tiles * p.splits);
    hipLaunchKernelGGL((i2s_decode_kernel<NT, 2>), dim3(grid), dim3(kBlock), 0, stream,
                       static_cast<const uint8_t*>(packed), w_scale, xq, x_scale, M, N, K, y, acc, partial, tickets,
                       p.splits, p.kb_per_split);
    return hipGetLastError();
}

}  // namespace

DecodePlan plan_i2s_decode(int64_t N, int64_t K) {
    DecodePlan p;
    const int nrg = (int)(N / kRowsPerGroup);
    p.nt = (nrg % 2 == 0) ? 2 : 1;
    p.tiles = nrg / p.nt;
    const int nkb = (int)((K + kI2sBlockK - 1) / kI2sBlockK);
    const int target_groups = 1024;                       // 4 work groups (16 waves) per CU
    int splits = (target_groups + p.tiles - 1) / p.tiles;
    splits = std::max(1, std::min(splits, std::max(1, nkb / kWaves)));
    p.kb_per_split = (nkb + splits - 1) / splits;
    p.splits = (nkb + p.kb_per_split - 1) / p.kb_per_split;
    return p;
}

size_t i2s_decode_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    (void)M;
    const DecodePlan p = plan_i2s_decode(N, K);
    if (p.splits <= 1) return 0;
    return (size_t)p.splits * 16 * (size_t)N * sizeof(int32_t) + (size_t)p.tiles * sizeof(unsigned);
}

hipError_t launch_i2s_decode(const void* packed, const float* w_scale, const int8_t* xq, const float* x_scale,
                             int M, int N, int K, float* y, int32_t* acc, void* ws, hipStream_t stream) {
    const DecodePlan p = plan_i2s_decode(N, K);
    if (p.nt == 2) return launch_nt<2>(p, packed, w_scale, xq, x_scale, M, N, K, y, acc, ws, stream);
    return launch_nt<1>(p, packed, w_scale, xq, x_scale, M, N, K, y, acc, ws, stream);
}

}  // namespace bitnet
