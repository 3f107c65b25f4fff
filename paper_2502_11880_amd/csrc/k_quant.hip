// Per-token absmax int8 activation quantisation (Sec. 2.1; Sec. 3.2.2 of the paper: the activations
// are quantised to int8 the way BitNet b1.58 trains, here with one scale per token row).
//
//   gamma_m = max_k |x[m, k]|, floored at 1e-5
//   s_m     = 127 / gamma_m                       (IEEE fp32 divide, round to nearest even)
//   xq      = clamp(rint(x * s_m), -128, 127)     (fp32 multiply, ties to even)
//   rowsum  = sum_k xq[m, k]                      (optional; exact int32)
//
// Many rows of up to 4096: one wave per row, reduced inside the wave.  Otherwise one work group per row.  The
// row is read once into registers (up to 16 float4 per lane), reduced to its absmax, then quantised from
// registers; rows too long for that take a second pass over memory.  HBM-bound: 4 bytes read and 1 byte
// written per element.
#include "bitnet_internal.hpp"

namespace bitnet {
namespace {

template <int BLOCK>
__device__ float block_max(float v, float* red) {
    v = wave_max(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    if (wave == 0) {
        float w = lane < BLOCK / 64 ? red[lane] : 0.0f;
        w = wave_max(w);
        if (lane == 0) red[0] = w;
    }
    __syncthreads();
    return red[0];
}

template <int BLOCK>
__device__ int block_sum(int v, int* red) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    int t = 0;
    for (int w = 0; w < BLOCK / 64; ++w) t += red[w];
    return t;
}

__device__ __forceinline__ int quant_one(float v, float s) {
    float r = rintf(v * s);
    r = fminf(fmaxf(r, -128.0f), 127.0f);
    return (int)r;
}

template <int BLOCK, int VPT>
__global__ __launch_bounds__(BLOCK) void quantize_rows_reg(const float* __restrict__ x, int K,
                                                           int8_t* __restrict__ xq, float* __restrict__ x_scale,
                                                           int32_t* __restrict__ x_rowsum) {
    __shared__ float red[BLOCK / 64];
    __shared__ int redi[BLOCK / 64];
    const size_t m = blockIdx.x;
    const float4* x4 = reinterpret_cast<const float4*>(x + m * (size_t)K);
    uint32_t* q4 = reinterpret_cast<uint32_t*>(xq + m * (size_t)K);
    const int K4 = K >> 2;
    float4 v[VPT];
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int idx = threadIdx.x + i * BLOCK;
        v[i] = idx < K4 ? x4[idx] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v[i].x), fabsf(v[i].y)), fmaxf(fabsf(v[i].z), fabsf(v[i].w))));
    }
    amax = block_max<BLOCK>(amax, red);
    const float s = 127.0f / fmaxf(amax, 1e-5f);
    if (threadIdx.x == 0) x_scale[m] = s;
    int sum = 0;
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int idx = threadIdx.x + i * BLOCK;
        if (idx < K4) {
            const uint32_t c = quant4(v[i], s);
            sum = byte_sum4(c, sum);
            q4[idx] = c;
        }
    }
    if (x_rowsum) {
        sum = block_sum<BLOCK>(sum, redi);
        if (threadIdx.x == 0) x_rowsum[m] = sum;
    }
}

// One wave per row (K <= 4096): the row in registers (up to 16 float4 per lane), absmax and code sum by DPP
// reductions inside the wave (no barrier), the codes packed four to a word by quant4.  A work group holds
// four independent rows.
template <int VPT>
__global__ __launch_bounds__(256) void quantize_rows_wave(const float* __restrict__ x, int64_t M, int K,
                                                          int8_t* __restrict__ xq, float* __restrict__ x_scale,
                                                          int32_t* __restrict__ x_rowsum) {
    const int lane = threadIdx.x & 63;
    const int64_t m = (int64_t)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (m >= M) return;
    const float4* x4 = reinterpret_cast<const float4*>(x + m * (size_t)K);
    uint32_t* q4 = reinterpret_cast<uint32_t*>(xq + m * (size_t)K);
    const int K4 = K >> 2;
    float4 v[VPT];
    float amax = 0.0f;
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int idx = lane + 64 * i;
        v[i] = idx < K4 ? x4[idx] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v[i].x), fabsf(v[i].y)), fmaxf(fabsf(v[i].z), fabsf(v[i].w))));
    }
    amax = wave_max_all(amax);
    const float s = 127.0f / fmaxf(amax, 1e-5f);
    int sum = 0;
#pragma unroll
    for (int i = 0; i < VPT; ++i) {
        const int idx = lane + 64 * i;
        if (idx < K4) {
            const uint32_t c = quant4(v[i], s);
            sum = byte_sum4(c, sum);
            q4[idx] = c;
        }
    }
    if (lane == 0) x_scale[m] = s;
    if (x_rowsum) {
        sum = wave_sum_all(sum);
        if (lane == 0) x_rowsum[m] = sum;
    }
}

// Any K: two passes over the row.
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void quantize_rows_2pass(const float* __restrict__ x, int K,
                                                             int8_t* __restrict__ xq, float* __restrict__ x_scale,
                                                             int32_t* __restrict__ x_rowsum) {
    __shared__ float red[BLOCK / 64];
    __shared__ int redi[BLOCK / 64];
    const size_t m = blockIdx.x;
    const float* xr = x + m * (size_t)K;
    int8_t* qr = xq + m * (size_t)K;
    float amax = 0.0f;
    for (int i = threadIdx.x; i < K; i += BLOCK) amax = fmaxf(amax, fabsf(xr[i]));
    amax = block_max<BLOCK>(amax, red);
    const float s = 127.0f / fmaxf(amax, 1e-5f);
    if (threadIdx.x == 0) x_scale[m] = s;
    int sum = 0;
    for (int i = threadIdx.x; i < K; i += BLOCK) {
        const int c = quant_one(xr[i], s);
        sum += c;
        qr[i] = (int8_t)c;
    }
    if (x_rowsum) {
        sum = block_sum<BLOCK>(sum, redi);
        if (threadIdx.x == 0) x_rowsum[m] = sum;
    }
}

template <int BLOCK>
hipError_t launch_block(const float* x, int64_t M, int64_t K, int8_t* xq, float* x_scale, int32_t* x_rowsum,
                        hipStream_t stream) {
    const dim3 grid((unsigned)M), block(BLOCK);
    const int64_t K4 = K / 4;
    if (K % 4 != 0 || K4 > 16 * BLOCK) {
        hipLaunchKernelGGL(quantize_rows_2pass<BLOCK>, grid, block, 0, stream, x, (int)K, xq, x_scale, x_rowsum);
    } else if (K4 <= BLOCK) {
        hipLaunchKernelGGL((quantize_rows_reg<BLOCK, 1>), grid, block, 0, stream, x, (int)K, xq, x_scale, x_rowsum);
    } else if (K4 <= 2 * BLOCK) {
        hipLaunchKernelGGL((quantize_rows_reg<BLOCK, 2>), grid, block, 0, stream, x, (int)K, xq, x_scale, x_rowsum);
    } else if (K4 <= 4 * BLOCK) {
        hipLaunchKernelGGL((quantize_rows_reg<BLOCK, 4>), grid, block, 0, stream, x, (int)K, xq, x_scale, x_rowsum);
    } else if (K4 <= 8 * BLOCK) {
        hipLaunchKernelGGL((quantize_rows_reg<BLOCK, 8>), grid, block, 0, stream, x, (int)K, xq, x_scale, x_rowsum);
    } else {
        hipLaunchKernelGGL((quantize_rows_reg<BLOCK, 16>), grid, block, 0, stream, x, (int)K, xq, x_scale, x_rowsum);
    }
    return hipGetLastError();
}

template <int VPT>
hipError_t launch_wave(const float* x, int64_t M, int64_t K, int8_t* xq, float* x_scale, int32_t* x_rowsum,
                       hipStream_t stream) {
    hipLaunchKernelGGL((quantize_rows_wave<VPT>), dim3((unsigned)((M + 3) / 4)), dim3(256), 0, stream, x, M, (int)K, xq,
                       x_scale, x_rowsum);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize_act(const float* x, int64_t M, int64_t K, int8_t* xq, float* x_scale,
                               int32_t* x_rowsum, hipStream_t stream) {
    // Few rows: wide groups so one row is spread over many lanes.  Many rows of up to 4096: one wave each;
    // longer rows: one 256-lane group each.
    if (M <= 64) return launch_block<1024>(x, M, K, xq, x_scale, x_rowsum, stream);
    if (K % 4 == 0 && K <= 1024) return launch_wave<4>(x, M, K, xq, x_scale, x_rowsum, stream);
    if (K % 4 == 0 && K <= 2048) return launch_wave<8>(x, M, K, xq, x_scale, x_rowsum, stream);
    if (K % 4 == 0 && K <= 4096) return launch_wave<16>(x, M, K, xq, x_scale, x_rowsum, stream);
    return launch_block<256>(x, M, K, xq, x_scale, x_rowsum, stream);
}

}  // namespace bitnet
