// Prefill GEMM for the I2_S layout (M > 16 tokens): ternary x int8 accumulation (Eq. 1) as a dense int8
// contraction on v_mfma_i32_16x16x64_i8, with the dequantisation epilogue fused.  The paper leaves prefill
// open (Sec. "Limitations": prefill is compute-bound, so its CPU methods do not apply); this kernel is the
// MFMA-bound design for it.
//
// Tiles: a work group of 4 waves computes a 128-token x 128-row output tile; each wave owns 64 x 64 (4 x 4
// MFMA tiles).  K advances in 256-k stages, the I2_S block size, so the packed weights of one row group and
// stage are one contiguous KiB: every lane loads its 16 bytes straight into registers (four MFMA B words) and
// unpacks them there, so the weights never pass through LDS.  The int8 activation tile (128 x 256) is staged
// in LDS with rows padded to 272 bytes, so the 16 rows an A operand reads fall on distinct banks.  The next
// stage's global loads are issued before the current stage's MFMAs.
//
// The codes are t + 1; sum_k xq[m, k] over the whole K is accumulated by the threads that stage the
// activation rows and subtracted in the epilogue (exact integers).
#include "bitnet_internal.hpp"

namespace bitnet {
namespace {

constexpr int kBM = 128, kBN = 128, kBK = 256;
constexpr int kThreads = 256;
constexpr int kARow = kBK + 16;            // padded LDS row of the activation tile

__device__ __forceinline__ v4i unpack_codes(uint32_t w) {
    v4i b;
    b.x = (int)(w & 0x03030303u);
    b.y = (int)((w >> 2) & 0x03030303u);
    b.z = (int)((w >> 4) & 0x03030303u);
    b.w = (int)((w >> 6) & 0x03030303u);
    return b;
}

__device__ __forceinline__ uint32_t word_of(const v4u& v, int j) {
    return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
}

__device__ __forceinline__ int byte_sum(const v4i& v) {
    const int ones = 0x01010101;
    int s = __builtin_amdgcn_sdot4(v.x, ones, 0, false);
    s = __builtin_amdgcn_sdot4(v.y, ones, s, false);
    s = __builtin_amdgcn_sdot4(v.z, ones, s, false);
    return __builtin_amdgcn_sdot4(v.w, ones, s, false);
}

__global__ __launch_bounds__(kThreads) void i2s_prefill_kernel(
    const uint8_t* __restrict__ packed, const float* __restrict__ w_scale, const int8_t* __restrict__ xq,
    const float* __restrict__ x_scale, int M, int N, int K, float* __restrict__ y, int32_t* __restrict__ acc_out) {
    __shared__ __align__(16) int8_t As[kBM * kARow];
    __shared__ int rowsum_s[kBM];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int q = lane >> 4, r = lane & 15;
    const int tiles_m = (M + kBM - 1) / kBM;
    const int L = xcd_logical_id(blockIdx.x, gridDim.x);
    const int tm = L % tiles_m, tn = L / tiles_m;       // neighbours share a weight tile
    const int m0 = tm * kBM, n0 = tn * kBN;
    const int nkb = (K + kBK - 1) / kBK;
    const int nfull = K / kBK;
    const int nrg = N / kRowsPerGroup;
    const size_t rg_bytes = (size_t)4 * K;

    // activation staging: thread -> (row, half); 8 x 16 bytes of one row per stage
    const int a_row = tid >> 1, a_half = tid & 1;
    const bool a_valid = m0 + a_row < M;
    const int8_t* a_src = xq + (size_t)(a_valid ? m0 + a_row : 0) * K + 128 * a_half;
    int8_t* a_dst = As + a_row * kARow + 128 * a_half;

    // weight row groups of this wave
    int rgs[4];
    bool rg_ok[4];
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) {
        rgs[ni] = n0 / kRowsPerGroup + 4 * wn + ni;
        rg_ok[ni] = rgs[ni] < nrg;
    }

    const v4i zero = {0, 0, 0, 0};
    v4i acc[4][4];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = zero;
    int rs = 0;

    v4i a_reg[8];
    v4u b_next[4], b_cur[4];

    auto load_stage = [&](int kb) {
        const int T = kb < nfull ? 4 : (K - nfull * kBK) / kSubK;   // 64-k sub-tiles in this stage
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int koff = 128 * a_half + 16 * i;
            a_reg[i] = (a_valid && koff < 64 * T) ? *reinterpret_cast<const v4i*>(a_src + (size_t)kb * kBK + 16 * i)
                                                  : zero;
        }
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
            v4u w = {0u, 0u, 0u, 0u};
            if (rg_ok[ni]) {
                const uint8_t* p = packed + (size_t)rgs[ni] * rg_bytes + (size_t)kb * 1024;
                if (T == 4) {
                    w = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p + 16 * lane));
                } else {
                    const uint32_t* pw = reinterpret_cast<const uint32_t*>(p + 4 * T * lane);
                    w.x = pw[0];
                    if (T > 1) w.y = pw[1];
                    if (T > 2) w.z = pw[2];
                }
            }
            b_next[ni] = w;
        }
    };
    auto store_stage = [&]() {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            *reinterpret_cast<v4i*>(a_dst + 16 * i) = a_reg[i];
            rs += byte_sum(a_reg[i]);
        }
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) b_cur[ni] = b_next[ni];
    };

    load_stage(0);
    store_stage();
    __syncthreads();
    for (int kb = 0; kb < nkb; ++kb) {
        const int T = kb < nfull ? 4 : (K - nfull * kBK) / kSubK;
        if (kb + 1 < nkb) load_stage(kb + 1);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (j < T) {
                v4i a[4];
#pragma unroll
                for (int mi = 0; mi < 4; ++mi)
                    a[mi] = *reinterpret_cast<const v4i*>(As + (64 * wm + 16 * mi + r) * kARow + kSubK * j + 16 * q);
#pragma unroll
                for (int ni = 0; ni < 4; ++ni) {
                    const v4i b = unpack_codes(word_of(b_cur[ni], j));
#pragma unroll
                    for (int mi = 0; mi < 4; ++mi)
                        acc[mi][ni] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[mi], b, acc[mi][ni], 0, 0, 0);
                }
            }
        }
        __syncthreads();
        if (kb + 1 < nkb) {
            store_stage();
            __syncthreads();
        }
    }

    // token sums of this tile's rows: the two halves of each row
    rs += __shfl_xor(rs, 1, 64);
    if (a_half == 0) rowsum_s[a_row] = rs;
    __syncthreads();

    const float beta = *w_scale;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int ml = 64 * wm + 16 * mi + 4 * q + v;      // D row 4*(lane/16) + v
            const int m = m0 + ml;
            if (m >= M) continue;
            const int rsum = rowsum_s[ml];
            const float sc = beta / x_scale[m];
#pragma unroll
            for (int ni = 0; ni < 4; ++ni) {
                if (!rg_ok[ni]) continue;
                const int n = rgs[ni] * kRowsPerGroup + r;      // D column lane % 16
                const int val = acc[mi][ni][v] - rsum;
                y[(size_t)m * N + n] = (float)val * sc;
                if (acc_out) acc_out[(size_t)m * N + n] = val;
            }
        }
    }
}

}  // namespace

hipError_t launch_i2s_prefill(const void* packed, const float* w_scale, const int8_t* xq, const float* x_scale,
                              int M, int N, int K, float* y, int32_t* acc, hipStream_t stream) {
    const unsigned tiles = (unsigned)(((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN));
    hipLaunchKernelGGL(i2s_prefill_kernel, dim3(tiles), dim3(kThreads), 0, stream,
                       static_cast<const uint8_t*>(packed), w_scale, xq, x_scale, M, N, K, y, acc);
    return hipGetLastError();
}

}  // namespace bitnet
