// Internal declarations shared by the library's translation units (host launchers + device helpers).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace bitnet {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

constexpr int kRowsPerGroup = 16;     // weight rows per MFMA tile (both layouts)
constexpr int kSubK = 64;             // k per 16x16x64 int8 MFMA
constexpr int kI2sBlockK = 256;       // I2_S block: up to four 64-k sub-tiles, 1 KiB per row group
constexpr int kTl2BlockK = 384;       // TL2 block BK3: 128 triples per row
constexpr int kNumXcd = 8;            // MI355X: 8 accelerator dies, work groups dealt round-robin

// ------------------------------------------------------------------------------------------------
// Device helpers
// ------------------------------------------------------------------------------------------------

// Work groups are dealt to the XCDs round-robin by id.  Renumber them so that each XCD owns one
// contiguous range of logical ids; neighbouring tiles (split-K siblings) then share an L2.
__device__ __forceinline__ int xcd_logical_id(int bid, int nblocks) {
    const int per = nblocks / kNumXcd, extra = nblocks % kNumXcd;
    const int xcd = bid % kNumXcd, idx = bid / kNumXcd;
    return xcd * per + (xcd < extra ? xcd : extra) + idx;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

// ------------------------------------------------------------------------------------------------
// Host launchers (each returns the launch status; shapes were validated by the caller)
// ------------------------------------------------------------------------------------------------
hipError_t launch_quantize_act(const float* x, int64_t M, int64_t K, int8_t* xq, float* x_scale,
                               hipStream_t stream);

size_t pack_workspace_bytes();
hipError_t launch_pack(int layout, const float* W, int64_t N, int64_t K, void* packed, float* w_scale,
                       void* ws, hipStream_t stream);

int i2s_decode_waves(int64_t K);
hipError_t launch_i2s_decode(const void* packed, const float* w_scale, const int8_t* xq,
                             const float* x_scale, int M, int N, int K, float* y, int32_t* acc,
                             hipStream_t stream);

hipError_t launch_i2s_prefill(const void* packed, const float* w_scale, const int8_t* xq, const float* x_scale,
                              int M, int N, int K, float* y, int32_t* acc, hipStream_t stream);

constexpr int kElutMaxTokens = 8;     // tokens per ELUT launch
int tl2_elut_waves(int M);
size_t tl2_elut_lds_bytes(int M);
hipError_t launch_tl2_elut_decode(const void* packed, const float* w_scale, const int8_t* xq,
                                  const float* x_scale, int M, int N, int K, float* y, int32_t* acc,
                                  hipStream_t stream);
hipError_t launch_elut_tables(const int8_t* xq, int M, int K, int16_t* lut, int16_t* lut1, hipStream_t stream);

}  // namespace bitnet
