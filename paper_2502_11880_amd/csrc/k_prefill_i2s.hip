// Prefill GEMM for the I2_S layout (M > 16 tokens): ternary x int8 accumulation (Eq. 1) as a dense int8
// contraction on v_mfma_i32_32x32x32_i8, with the dequantisation epilogue fused.  The paper leaves prefill
// open (Sec. "Limitations": prefill is compute-bound, so its CPU methods do not apply); this kernel is the
// MFMA-bound design for it.  (On gfx950 the 32x32x32 int8 MFMA sustains about twice the rate of the 16x16x64
// one, so the contraction uses the former.)
//
// Tiles: a work group of 4 waves computes a 128-token x 128-row output tile; each wave owns 64 x 64 (2 x 2
// MFMA tiles of 32 x 32).  K advances in 256-k stages, the I2_S block size, so the packed weights of one row
// group and stage are one contiguous KiB.  Lane (j, h) of a wave (j = lane % 32, h = lane / 32) needs, for
// its weight row j, the 16 codes of k-step s at k = 32 s + 16 h: these are word s/2 of the layout's lane chunk
// q = 2 (s % 2) + h, so each lane loads two 16-byte chunks per 32-row tile per stage straight into registers
// and unpacks them there; the weights never pass through LDS.  The int8 activation tile (128 x 256) is
// staged in LDS with rows padded to 272 bytes.  The next stage's global loads are issued before the current
// stage's MFMAs.
//
// The codes are t + 1: sum_k xq[m, k] is subtracted in the epilogue, either from x_rowsum (written by the
// quantiser) or accumulated here by the threads that stage the activation rows.
#include "bitnet_internal.hpp"

namespace bitnet {
namespace {

typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBN = 128, kBK = 256;
constexpr int kThreads = 256;
constexpr int kARow = kBK + 16;            // padded LDS row of the activation tile

__device__ __forceinline__ int byte_sum(const v4i& v) {
    const int ones = 0x01010101;
    int s = __builtin_amdgcn_sdot4(v.x, ones, 0, false);
    s = __builtin_amdgcn_sdot4(v.y, ones, s, false);
    s = __builtin_amdgcn_sdot4(v.z, ones, s, false);
    return __builtin_amdgcn_sdot4(v.w, ones, s, false);
}

template <bool HAS_RS>
__global__ __launch_bounds__(kThreads) void i2s_prefill_kernel(
    const uint8_t* __restrict__ packed, const float* __restrict__ w_scale, const int8_t* __restrict__ xq,
    const float* __restrict__ x_scale, const int32_t* __restrict__ x_rowsum, int M, int N, int K,
    float* __restrict__ y, int32_t* __restrict__ acc_out) {
    __shared__ __align__(16) int8_t As[kBM * kARow];
    __shared__ int rowsum_s[kBM];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int j32 = lane & 31, h = lane >> 5;
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

    // weight row group and lane chunk of each 32-row tile of this wave
    int rg[2];
    bool rg_ok[2];
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
        rg[ni] = n0 / kRowsPerGroup + 4 * wn + 2 * ni + (j32 >> 4);
        rg_ok[ni] = rg[ni] < nrg;
    }
    const int r16 = j32 & 15;

    const v4i zero4 = {0, 0, 0, 0};
    v16i acc[2][2];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) acc[mi][ni] = v16i{};
    int rs = 0;

    v4i a_reg[8];
    v4u b_next[2][2], b_cur[2][2];     // [tile][chunk: q = h, q = 2 + h]

    auto load_stage = [&](int kb) {
        const int T = kb < nfull ? 4 : (K - nfull * kBK) / kSubK;   // 64-k sub-tiles in this stage
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int koff = 128 * a_half + 16 * i;
            a_reg[i] = (a_valid && koff < 64 * T) ? *reinterpret_cast<const v4i*>(a_src + (size_t)kb * kBK + 16 * i)
                                                  : zero4;
        }
#pragma unroll
        for (int ni = 0; ni < 2; ++ni) {
#pragma unroll
            for (int c = 0; c < 2; ++c) {
                v4u w = {0u, 0u, 0u, 0u};
                if (rg_ok[ni]) {
                    const int ql = 16 * (2 * c + h) + r16;              // lane of the layout's chunk
                    const uint8_t* p = packed + (size_t)rg[ni] * rg_bytes + (size_t)kb * 1024;
                    if (T == 4) {
                        w = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p + 16 * ql));
                    } else {
                        const uint32_t* pw = reinterpret_cast<const uint32_t*>(p + 4 * T * ql);
                        w.x = pw[0];
                        if (T > 1) w.y = pw[1];
                        if (T > 2) w.z = pw[2];
                    }
                }
                b_next[ni][c] = w;
            }
        }
    };
    auto store_stage = [&]() {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            *reinterpret_cast<v4i*>(a_dst + 16 * i) = a_reg[i];
            if (!HAS_RS) rs += byte_sum(a_reg[i]);
        }
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
#pragma unroll
            for (int c = 0; c < 2; ++c) b_cur[ni][c] = b_next[ni][c];
    };

    load_stage(0);
    store_stage();
    __syncthreads();
    for (int kb = 0; kb < nkb; ++kb) {
        const int T = kb < nfull ? 4 : (K - nfull * kBK) / kSubK;
        if (kb + 1 < nkb) load_stage(kb + 1);
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            if (s < 2 * T) {
                v4i a[2];
#pragma unroll
                for (int mi = 0; mi < 2; ++mi)
                    a[mi] = *reinterpret_cast<const v4i*>(As + (64 * wm + 32 * mi + j32) * kARow + 32 * s + 16 * h);
#pragma unroll
                for (int ni = 0; ni < 2; ++ni) {
                    const v4i b = unpack_codes(word_of(b_cur[ni][s & 1], s >> 1));
#pragma unroll
                    for (int mi = 0; mi < 2; ++mi)
                        acc[mi][ni] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[mi], b, acc[mi][ni], 0, 0, 0);
                }
            }
        }
        __syncthreads();
        if (kb + 1 < nkb) {
            store_stage();
            __syncthreads();
        }
    }

    if (HAS_RS) {
        if (tid < kBM) rowsum_s[tid] = (m0 + tid < M) ? x_rowsum[m0 + tid] : 0;
    } else {
        rs += __shfl_xor(rs, 1, 64);                     // the two halves of each row
        if (a_half == 0) rowsum_s[a_row] = rs;
    }
    __syncthreads();

    // D element v of lane (j, h): row 8 * (v / 4) + 4 * h + v % 4, column j.
    const float beta = *w_scale;
#pragma unroll
    for (int mi = 0; mi < 2; ++mi) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int ml = 64 * wm + 32 * mi + 8 * (v >> 2) + 4 * h + (v & 3);
            const int m = m0 + ml;
            if (m >= M) continue;
            const int rsum = rowsum_s[ml];
            const float sc = beta / x_scale[m];
#pragma unroll
            for (int ni = 0; ni < 2; ++ni) {
                if (!rg_ok[ni]) continue;
                const int n = rg[ni] * kRowsPerGroup + r16;
                const int val = acc[mi][ni][v] - rsum;
                y[(size_t)m * N + n] = (float)val * sc;
                if (acc_out) acc_out[(size_t)m * N + n] = val;
            }
        }
    }
}

}  // namespace

hipError_t launch_i2s_prefill(const void* packed, const float* w_scale, const int8_t* xq, const float* x_scale,
                              const int32_t* x_rowsum, int M, int N, int K, float* y, int32_t* acc,
                              hipStream_t stream) {
    const unsigned tiles = (unsigned)(((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN));
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    if (x_rowsum)
        hipLaunchKernelGGL(i2s_prefill_kernel<true>, dim3(tiles), dim3(kThreads), 0, stream, pk, w_scale, xq, x_scale,
                           x_rowsum, M, N, K, y, acc);
    else
        hipLaunchKernelGGL(i2s_prefill_kernel<false>, dim3(tiles), dim3(kThreads), 0, stream, pk, w_scale, xq,
                           x_scale, x_rowsum, M, N, K, y, acc);
    return hipGetLastError();
}

}  // namespace bitnet
