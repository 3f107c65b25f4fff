// Per-token absmax int8 activation quantisation (Sec. 2.1; Sec. 3.2.2 of the paper: the activations
// are quantised to int8 the way BitNet b1.58 trains, here with one scale per token row).
//
//   gamma_m = max_k |x[m, k]|, floored at 1e-5
//   s_m     = 127 / gamma_m                       (IEEE fp32 divide, round to nearest even)
//   xq      = clamp(rint(x * s_m), -128, 127)     (fp32 multiply, ties to even)
//
// One work group per token row: a first pass finds the absmax, a second pass (an L2 hit) writes the
// codes.  HBM-bound: 4 bytes read and 1 byte written per element.
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

__device__ __forceinline__ int quant_one(float v, float s) {
    float r = rintf(v * s);
    r = fminf(fmaxf(r, -128.0f), 127.0f);
    return (int)r;
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void quantize_rows(const float* __restrict__ x, int K,
                                                       int8_t* __restrict__ xq, float* __restrict__ x_scale) {
    __shared__ float red[BLOCK / 64];
    const size_t m = blockIdx.x;
    const float* xr = x + m * (size_t)K;
    int8_t* qr = xq + m * (size_t)K;
    const bool vec = (K & 3) == 0;
    const int K4 = vec ? K >> 2 : 0;

    float amax = 0.0f;
    if (vec) {
        const float4* x4 = reinterpret_cast<const float4*>(xr);
        for (int i = threadIdx.x; i < K4; i += BLOCK) {
            const float4 v = x4[i];
            amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w))));
        }
    } else {
        for (int i = threadIdx.x; i < K; i += BLOCK) amax = fmaxf(amax, fabsf(xr[i]));
    }
    amax = block_max<BLOCK>(amax, red);
    const float gamma = fmaxf(amax, 1e-5f);
    const float s = 127.0f / gamma;
    if (threadIdx.x == 0) x_scale[m] = s;

    if (vec) {
        const float4* x4 = reinterpret_cast<const float4*>(xr);
        uint32_t* q4 = reinterpret_cast<uint32_t*>(qr);
        for (int i = threadIdx.x; i < K4; i += BLOCK) {
            const float4 v = x4[i];
            const uint32_t w = (uint32_t)(quant_one(v.x, s) & 0xFF) |
                               ((uint32_t)(quant_one(v.y, s) & 0xFF) << 8) |
                               ((uint32_t)(quant_one(v.z, s) & 0xFF) << 16) |
                               ((uint32_t)(quant_one(v.w, s) & 0xFF) << 24);
            q4[i] = w;
        }
    } else {
        for (int i = threadIdx.x; i < K; i += BLOCK) qr[i] = (int8_t)quant_one(xr[i], s);
    }
}

}  // namespace

hipError_t launch_quantize_act(const float* x, int64_t M, int64_t K, int8_t* xq, float* x_scale,
                               hipStream_t stream) {
    // Few rows: wide groups so one row is spread over many lanes.  Many rows: one 256-lane group each.
    if (M <= 64) {
        hipLaunchKernelGGL(quantize_rows<1024>, dim3((unsigned)M), dim3(1024), 0, stream, x, (int)K, xq,
                           x_scale);
    } else {
        hipLaunchKernelGGL(quantize_rows<256>, dim3((unsigned)M), dim3(256), 0, stream, x, (int)K, xq,
                           x_scale);
    }
    return hipGetLastError();
}

}  // namespace bitnet
