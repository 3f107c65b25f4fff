// Decode GEMV for the I2_S layout (M <= 16 tokens): ternary x int8 accumulation (Eq. 1) on int8 MFMA,
// with the dequantisation epilogue fused.
//
// Weights are HBM-bound: each packed byte is read exactly once, with 16-byte non-temporal loads, one
// contiguous KiB per wave per 256-k block.  A 32-bit word of lane (r, q) holds 16 codes c = t + 1 of
// row r; shifting by 2f and masking 0x03030303 gives the four int8 codes of k = 4f .. 4f+3, which is
// exactly the byte order of the matching activation word.  So the unpacked word feeds the B operand of
// v_mfma_i32_16x16x64_i8 directly (B column = weight row, A row = token; tokens beyond M are zero).
// The codes carry a +1 offset, removed by subtracting sum_k xq[m, k]: read from x_rowsum (written by the
// quantiser) when given, otherwise taken with a second MFMA against an all-ones B over the same k.
//
// Work split: one work group per 16-row group, holding the whole K.  Its 4, 8 or 16 waves take every
// WAVES-th 256-k block, issue their weight loads U blocks at a time (a GEMV of a few MB is latency-bound:
// one DRAM round trip should cover it) and reduce through LDS; wave 0 applies the epilogue.  No work group
// depends on another, so no device-wide fence is needed (an agent-scope release writes back the whole L2
// of the XCD, which costs more than these GEMVs).  One launch may cover several weights that share the
// activation (the grid concatenates their row groups).
//
// Single-token fused variant: the work group also quantises the activation row itself (Sec. 2.1): it loads
// the fp32 row into registers before issuing its weight loads, reduces the absmax through LDS, and writes
// the codes to LDS, where the MFMA A operands are read; the sum of the codes replaces x_rowsum.  The weight
// loads stay in flight during all of this.
#include "bitnet_internal.hpp"

namespace bitnet {
namespace {

__device__ __forceinline__ int q8(float v, float s) {
    return (int)fminf(fmaxf(rintf(v * s), -128.0f), 127.0f);
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Which weight and row group this work group serves.
__device__ __forceinline__ void locate(const FusedLinears& L, int bid, int& li, int& rg) {
    li = 0;
    while (li + 1 < L.count && bid >= L.rg_start[li + 1]) ++li;
    rg = bid - L.rg_start[li];
}

// Multiply-accumulate of one 256-k block (T sub-tiles of 64): A from `arow` (global or LDS), B words from `w`.
template <bool HAS_RS>
__device__ __forceinline__ void block_mac(const int8_t* arow, int kb, int T, bool a_on, const v4u& w, v4i& acc,
                                          v4i& rowsum) {
    const v4i zero = {0, 0, 0, 0};
    const v4i ones = {0x01010101, 0x01010101, 0x01010101, 0x01010101};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (j < T) {
            const v4i a = a_on ? *reinterpret_cast<const v4i*>(arow + kb * kI2sBlockK + kSubK * j) : zero;
            acc = mfma16x16x64(a, unpack_codes(word_of(w, j)), acc);
            if (!HAS_RS) rowsum = mfma16x16x64(a, ones, rowsum);
        }
    }
}

// The weight words of block kb for this lane (a short last block has T words 4*T bytes apart).
__device__ __forceinline__ v4u block_words(const uint8_t* wbase, int kb, int nfull, int T, int lane) {
    if (kb < nfull) return load_stream16(wbase + (size_t)kb * 1024 + 16 * lane);
    v4u w = {0u, 0u, 0u, 0u};
    const uint32_t* p = reinterpret_cast<const uint32_t*>(wbase + (size_t)kb * 1024 + 4 * T * lane);
    w.x = p[0];
    if (T > 1) w.y = p[1];
    if (T > 2) w.z = p[2];
    return w;
}

template <int WAVES, int U, bool HAS_RS>
__global__ __launch_bounds__(64 * WAVES) void i2s_decode_kernel(FusedLinears L, const int8_t* __restrict__ xq,
                                                                const float* __restrict__ x_scale,
                                                                const int32_t* __restrict__ x_rowsum, int M, int K) {
    __shared__ v4i red[WAVES][64];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int li, rg;
    locate(L, xcd_logical_id(blockIdx.x, gridDim.x), li, rg);
    const int N = L.N[li];
    const int nkb = (K + kI2sBlockK - 1) / kI2sBlockK;
    const int nfull = K / kI2sBlockK;
    const int Tlast = nkb > nfull ? (K - nfull * kI2sBlockK) / kSubK : 4;
    const int q = lane >> 4, r = lane & 15;
    const bool a_on = r < M;                        // A operand: row = token r, 16 k per lane group q
    const int8_t* arow = xq + (size_t)(a_on ? r : 0) * K + 16 * q;
    const uint8_t* wbase = L.packed[li] + (size_t)rg * 4 * K;
    const v4i zero = {0, 0, 0, 0};

    v4i acc = zero, rowsum = zero;
    for (int kb = wave; kb < nkb; kb += WAVES * U) {
        v4u wv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kbu = kb + WAVES * u;
            if (kbu < nkb) wv[u] = block_words(wbase, kbu, nfull, kbu < nfull ? 4 : Tlast, lane);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kbu = kb + WAVES * u;
            if (kbu < nkb) block_mac<HAS_RS>(arow, kbu, kbu < nfull ? 4 : Tlast, a_on, wv[u], acc, rowsum);
        }
    }

    red[wave][lane] = acc - rowsum;
    __syncthreads();
    if (wave != 0) return;
    acc = red[0][lane];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) acc += red[w][lane];

    // Output element v of lane l is D[row 4*(l/16) + v][col l%16]: token m = 4q + v, weight row r.
    const float beta = *L.w_scale[li];
    float* y = L.y[li];
    int32_t* acc_out = L.acc[li];
    const int n = rg * kRowsPerGroup + r;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int m = 4 * q + v;
        if (m < M) {
            const float sc = beta / x_scale[m];
            const int val = HAS_RS ? acc[v] - x_rowsum[m] : acc[v];
            y[(size_t)m * N + n] = (float)val * sc;
            if (acc_out) acc_out[(size_t)m * N + n] = val;
        }
    }
}

// One token: quantise x (fp32 [K]) inside every work group, then the GEMV as above with A from LDS.
// XV float4 of the row per lane (XV * 4 * 64 * WAVES >= K); U blocks per wave in one batch.
template <int WAVES, int U, int XV>
__global__ __launch_bounds__(64 * WAVES) void i2s_decode_quant_kernel(FusedLinears L, const float* __restrict__ x,
                                                                      int K, int8_t* __restrict__ xq_out,
                                                                      float* __restrict__ s_out,
                                                                      int32_t* __restrict__ rs_out) {
    extern __shared__ __align__(16) int8_t xs[];      // K codes; later reused for the wave reduction
    __shared__ float redf[WAVES];
    __shared__ int redi[WAVES];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bid = xcd_logical_id(blockIdx.x, gridDim.x);
    int li, rg;
    locate(L, bid, li, rg);
    const int nkb = (K + kI2sBlockK - 1) / kI2sBlockK;
    const int nfull = K / kI2sBlockK;
    const int Tlast = nkb > nfull ? (K - nfull * kI2sBlockK) / kSubK : 4;
    const int q = lane >> 4, r = lane & 15;
    const uint8_t* wbase = L.packed[li] + (size_t)rg * 4 * K;
    const int K4 = K >> 2;

    // 1. the activation row into registers, then this wave's weights (all blocks of the first batch)
    const float4* x4 = reinterpret_cast<const float4*>(x);
    float4 xv[XV];
#pragma unroll
    for (int i = 0; i < XV; ++i) {
        const int e = tid + i * 64 * WAVES;
        xv[i] = e < K4 ? x4[e] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
    v4u wv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int kbu = wave + WAVES * u;
        if (kbu < nkb) wv[u] = block_words(wbase, kbu, nfull, kbu < nfull ? 4 : Tlast, lane);
    }

    // 2. absmax, scale, codes into LDS and their sum
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < XV; ++i)
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(xv[i].x), fabsf(xv[i].y)), fmaxf(fabsf(xv[i].z), fabsf(xv[i].w))));
    amax = wave_max(amax);
    if (lane == 0) redf[wave] = amax;
    __syncthreads();
    amax = redf[0];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) amax = fmaxf(amax, redf[w]);
    const float s = 127.0f / fmaxf(amax, 1e-5f);
    int sum = 0;
#pragma unroll
    for (int i = 0; i < XV; ++i) {
        const int e = tid + i * 64 * WAVES;
        if (e < K4) {
            const int c0 = q8(xv[i].x, s), c1 = q8(xv[i].y, s), c2 = q8(xv[i].z, s), c3 = q8(xv[i].w, s);
            sum += c0 + c1 + c2 + c3;
            reinterpret_cast<uint32_t*>(xs)[e] = (uint32_t)(c0 & 0xFF) | ((uint32_t)(c1 & 0xFF) << 8) |
                                                 ((uint32_t)(c2 & 0xFF) << 16) | ((uint32_t)(c3 & 0xFF) << 24);
        }
    }
    sum = wave_sum(sum);
    if (lane == 0) redi[wave] = sum;
    __syncthreads();
    int rowsum = 0;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) rowsum += redi[w];
    if (bid == 0) {
        for (int e = tid; e < K4; e += 64 * WAVES)
            reinterpret_cast<uint32_t*>(xq_out)[e] = reinterpret_cast<const uint32_t*>(xs)[e];
        if (tid == 0) {
            s_out[0] = s;
            rs_out[0] = rowsum;
        }
    }

    // 3. the GEMV: token 0 only (lanes r == 0 carry A)
    const bool a_on = r == 0;
    const int8_t* arow = xs + 16 * q;
    v4i acc = {0, 0, 0, 0}, unused = {0, 0, 0, 0};
    for (int kb = wave; kb < nkb; kb += WAVES * U) {
        if (kb != wave) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int kbu = kb + WAVES * u;
                if (kbu < nkb) wv[u] = block_words(wbase, kbu, nfull, kbu < nfull ? 4 : Tlast, lane);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kbu = kb + WAVES * u;
            if (kbu < nkb) block_mac<true>(arow, kbu, kbu < nfull ? 4 : Tlast, a_on, wv[u], acc, unused);
        }
    }

    __syncthreads();                  // every wave is done reading the codes: reuse the LDS
    v4i* red = reinterpret_cast<v4i*>(xs);
    red[wave * 64 + lane] = acc;
    __syncthreads();
    if (wave != 0 || q != 0) return;
#pragma unroll
    for (int w = 1; w < WAVES; ++w) acc += red[w * 64 + lane];
    // token 0 is D row 0: element 0 of lanes 0..15
    const float beta = *L.w_scale[li];
    const int n = rg * kRowsPerGroup + r;
    const int val = acc.x - rowsum;
    L.y[li][n] = (float)val * (beta / s);
    if (L.acc[li]) L.acc[li][n] = val;
}

template <int WAVES, int U>
void launch_plain(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum, int M, int K,
                  hipStream_t stream) {
    const dim3 grid((unsigned)L.rg_start[L.count]), block(64 * WAVES);
    if (x_rowsum)
        hipLaunchKernelGGL((i2s_decode_kernel<WAVES, U, true>), grid, block, 0, stream, L, xq, x_scale, x_rowsum, M, K);
    else
        hipLaunchKernelGGL((i2s_decode_kernel<WAVES, U, false>), grid, block, 0, stream, L, xq, x_scale, x_rowsum, M,
                           K);
}

template <int WAVES>
void launch_plain_u(int U, const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum,
                    int M, int K, hipStream_t stream) {
    if (U <= 1) launch_plain<WAVES, 1>(L, xq, x_scale, x_rowsum, M, K, stream);
    else if (U <= 2) launch_plain<WAVES, 2>(L, xq, x_scale, x_rowsum, M, K, stream);
    else launch_plain<WAVES, 4>(L, xq, x_scale, x_rowsum, M, K, stream);
}

template <int WAVES, int U>
void launch_quant(const FusedLinears& L, const float* x, int K, int8_t* xq, float* s, int32_t* rs, hipStream_t stream) {
    const dim3 grid((unsigned)L.rg_start[L.count]), block(64 * WAVES);
    const size_t lds = i2s_decode_quant_lds_bytes(K, WAVES);
    const int xv = (K / 4 + 64 * WAVES - 1) / (64 * WAVES);
    if (xv <= 1)
        hipLaunchKernelGGL((i2s_decode_quant_kernel<WAVES, U, 1>), grid, block, lds, stream, L, x, K, xq, s, rs);
    else if (xv <= 2)
        hipLaunchKernelGGL((i2s_decode_quant_kernel<WAVES, U, 2>), grid, block, lds, stream, L, x, K, xq, s, rs);
    else if (xv <= 4)
        hipLaunchKernelGGL((i2s_decode_quant_kernel<WAVES, U, 4>), grid, block, lds, stream, L, x, K, xq, s, rs);
    else if (xv <= 8)
        hipLaunchKernelGGL((i2s_decode_quant_kernel<WAVES, U, 8>), grid, block, lds, stream, L, x, K, xq, s, rs);
    else
        hipLaunchKernelGGL((i2s_decode_quant_kernel<WAVES, U, 16>), grid, block, lds, stream, L, x, K, xq, s, rs);
}

template <int WAVES>
void launch_quant_u(int U, const FusedLinears& L, const float* x, int K, int8_t* xq, float* s, int32_t* rs,
                    hipStream_t stream) {
    if (U <= 1) launch_quant<WAVES, 1>(L, x, K, xq, s, rs, stream);
    else if (U <= 2) launch_quant<WAVES, 2>(L, x, K, xq, s, rs, stream);
    else if (U <= 4) launch_quant<WAVES, 4>(L, x, K, xq, s, rs, stream);
    else launch_quant<WAVES, 8>(L, x, K, xq, s, rs, stream);
}

}  // namespace

// Waves per work group and blocks per wave per batch.  All waves of a launch should be resident at once
// (about 4096 on 256 CUs at the register use of these kernels): take the widest group (16, 8 or 4 waves) that
// keeps the launch within that, and let each wave load all of its blocks in one batch where the register
// budget allows (max_u).
void decode_shape(int64_t groups, int64_t K, int max_u, int min_waves, int& waves, int& u) {
    const int nkb = (int)((K + kI2sBlockK - 1) / kI2sBlockK);
    waves = 4;
    if (groups * 16 <= 4096) waves = 16;
    else if (groups * 8 <= 4096) waves = 8;
    if (waves < min_waves) waves = min_waves;
    while (waves < 16 && (nkb + waves - 1) / waves > max_u) waves *= 2;   // long K: one batch per wave
    u = (nkb + waves - 1) / waves;
    if (u > max_u) u = max_u;
}

size_t i2s_decode_quant_lds_bytes(int64_t K, int waves) {
    const size_t red = (size_t)waves * 64 * sizeof(v4i);
    return (size_t)K > red ? (size_t)K : red;
}

hipError_t launch_i2s_decode(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum,
                             int M, int K, hipStream_t stream) {
    int waves, u;
    decode_shape(L.rg_start[L.count], K, 4, 4, waves, u);
    switch (waves) {
        case 4: launch_plain_u<4>(u, L, xq, x_scale, x_rowsum, M, K, stream); break;
        case 8: launch_plain_u<8>(u, L, xq, x_scale, x_rowsum, M, K, stream); break;
        default: launch_plain_u<16>(u, L, xq, x_scale, x_rowsum, M, K, stream); break;
    }
    return hipGetLastError();
}

hipError_t launch_i2s_decode_quant(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                                   int32_t* x_rowsum, hipStream_t stream) {
    // the row lives in registers: at most 16 float4 per lane
    const int min_waves = K <= 16384 ? 4 : K <= 32768 ? 8 : 16;
    int waves, u;
    decode_shape(L.rg_start[L.count], K, 8, min_waves, waves, u);
    if (waves == 16 && u > 4) u = 4;     // 16-wave groups get 128 registers per lane
    switch (waves) {
        case 4: launch_quant_u<4>(u, L, x, K, xq, x_scale, x_rowsum, stream); break;
        case 8: launch_quant_u<8>(u, L, x, K, xq, x_scale, x_rowsum, stream); break;
        default: launch_quant_u<16>(u, L, x, K, xq, x_scale, x_rowsum, stream); break;
    }
    return hipGetLastError();
}

}  // namespace bitnet
