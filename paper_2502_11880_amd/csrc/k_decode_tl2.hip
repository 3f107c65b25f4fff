// TL2 accumulation by element-wise table lookup (ELUT, Eq. 3; Algorithm "ELUT mpGEMM"; Algorithm TL2),
// with mirror consolidation (Sec. 3.1.1), signed-unsigned weight splitting (Sec. 3.1.2), the 1-bit sign
// operation of Eq. 5 and TL1 lookups for the block-fitting tail (Table 5).
//
// Tables.  For token m and triple g with activations (a0, a1, a2) the table holds the 14 sums
//   T[i] = d0(i)*a0 + d1(i)*a1 + d2(i)*a2,  i = 9*d0 + 3*d1 + d2 in 0..13 (balanced ternary, leading digit >= 0),
// as int16 in a 32-byte slot (entries 14 and 15 are zero).  A TL1 pair (b0, b1) gets the 9 sums
//   T1[i] = (i/3 - 1)*b0 + (i%3 - 1)*b1.
//
// Lookup.  A triple contributes (T[idx] XOR m) - m with m = -sign (Eq. 5 with the sign bit widened to a mask).
// Summed over a lane's 32 triples the "- m" terms are just the number of negative triples, popcount(sign word),
// so each lookup costs one XOR-add.
//
// Work split: one work group per 16-row group.  Each wave takes every WAVES-th 384-k block, builds the tables of
// that block's 128 triples for the M tokens in its own LDS slice, and looks up its 16 rows x 128 triples.  The
// slices of different q quarters are skewed by 32 bytes so the four quarters read disjoint LDS banks.  Waves
// reduce through LDS; wave 0 applies the epilogue.
#include "bitnet_internal.hpp"

#include <algorithm>

namespace bitnet {
namespace {

constexpr int kSlot = 32;                                   // bytes per triple (or pair) table
constexpr int kTokenStride = (kTl2BlockK / 3 + 4) * kSlot;  // 128 triples + 4 skew slots per token

__device__ __forceinline__ int skewed_slot(int g) { return g + (g >> 5); }

__device__ __forceinline__ uint32_t pack16(int lo, int hi) {
    return ((uint32_t)lo & 0xFFFFu) | ((uint32_t)hi << 16);
}

// The 14 mirror-consolidated sums of one triple, as 8 words (16 int16, the last two zero).
__device__ __forceinline__ void triple_table(int a0, int a1, int a2, uint32_t w[8]) {
    const int p = a0 - a1, q = a0 + a1, s = a1 - a2, t = a1 + a2;
    w[0] = pack16(0, a2);                 // 000, 00+
    w[1] = pack16(s, a1);                 // 0+-, 0+0
    w[2] = pack16(t, p - a2);             // 0++, +--
    w[3] = pack16(p, p + a2);             // +-0, +-+
    w[4] = pack16(a0 - a2, a0);           // +0-, +00
    w[5] = pack16(a0 + a2, q - a2);       // +0+, ++-
    w[6] = pack16(q, q + a2);             // ++0, +++
    w[7] = 0u;
}

// The 9 sums of one TL1 pair (Table 5 order), as 8 words.
__device__ __forceinline__ void pair_table(int b0, int b1, uint32_t w[8]) {
    w[0] = pack16(-b0 - b1, -b0);          // (-,-), (-,0)
    w[1] = pack16(-b0 + b1, -b1);          // (-,+), (0,-)
    w[2] = pack16(0, b1);                  // (0,0), (0,+)
    w[3] = pack16(b0 - b1, b0);            // (+,-), (+,0)
    w[4] = pack16(b0 + b1, 0);             // (+,+)
    w[5] = 0u;
    w[6] = 0u;
    w[7] = 0u;
}

__device__ __forceinline__ void store_table(uint8_t* slot, const uint32_t w[8]) {
    v4u lo = {w[0], w[1], w[2], w[3]}, hi = {w[4], w[5], w[6], w[7]};
    reinterpret_cast<v4u*>(slot)[0] = lo;
    reinterpret_cast<v4u*>(slot)[1] = hi;
}

__device__ __forceinline__ int lds_i16(const uint8_t* p) { return (int)*reinterpret_cast<const int16_t*>(p); }

template <int WAVES, int MT>
__global__ __launch_bounds__(64 * WAVES) void tl2_elut_decode_kernel(
    const uint8_t* __restrict__ packed, const float* __restrict__ w_scale, const int8_t* __restrict__ xq,
    const float* __restrict__ x_scale, int M, int N, int K, float* __restrict__ y, int32_t* __restrict__ acc_out) {
    extern __shared__ __align__(16) uint8_t lds[];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int q = lane >> 4, r = lane & 15;
    const int rg = xcd_logical_id(blockIdx.x, gridDim.x);
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    const int nblk = three / kTl2BlockK;
    const int units = (K - three) / kSubK;
    const uint8_t* idx_plane = packed;
    const uint8_t* sign_plane = packed + (size_t)N * (three / 6);
    const uint8_t* tail_plane = sign_plane + (size_t)N * (three / 24);
    uint8_t* lut = lds + (size_t)wave * M * kTokenStride;

    int acc[MT];                                 // MT >= M tokens; loops run to MT with uniform guards
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = 0;

    for (int blk = wave; blk < nblk; blk += WAVES) {
        const size_t tile = (size_t)rg * nblk + blk;
        const v4u iw = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(idx_plane + tile * 1024 + 16 * lane));
        const uint32_t sw = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(sign_plane + tile * 256 + 4 * lane));
        // tables of this block's 128 triples: lane builds triples lane and lane + 64
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            if (m >= M) break;
            const int8_t* a = xq + (size_t)m * K + (size_t)blk * kTl2BlockK;
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int g = lane + 64 * h;
                uint32_t w[8];
                triple_table(a[3 * g], a[3 * g + 1], a[3 * g + 2], w);
                store_table(lut + m * kTokenStride + skewed_slot(g) * kSlot, w);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        // Lookups without branches: tokens past M (MT > M) read token 0's tables and are never stored, so all
        // 32 x MT reads of a lane can be in flight together (a guarded read per triple waits for each one).
        const uint8_t* base = lut + skewed_slot(32 * q) * kSlot;
#pragma unroll
        for (int i = 0; i < 32; ++i) {
            const uint32_t word = i < 8 ? iw.x : i < 16 ? iw.y : i < 24 ? iw.z : iw.w;
            const int idx = (int)((word >> (4 * (i & 7))) & 15u);
            const int msk = -(int)((sw >> i) & 1u);
            const uint8_t* e = base + i * kSlot + 2 * idx;
#pragma unroll
            for (int m = 0; m < MT; ++m) acc[m] += lds_i16(e + (m < M ? m : 0) * kTokenStride) ^ msk;
        }
        const int nneg = __popc(sw);
#pragma unroll
        for (int m = 0; m < MT; ++m) acc[m] += nneg;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    }

    // TL1 tail (K mod 384 weights): handled by the wave after the last TL2 block.
    if (units > 0 && wave == nblk % WAVES) {
        for (int u = 0; u < units; ++u) {
            const uint32_t word = *reinterpret_cast<const uint32_t*>(
                tail_plane + ((size_t)rg * 64 * units + (size_t)lane * units + u) * 4);
            // pair tables of this unit's 32 pairs (k = three + 64u + 2p), lanes 0..31
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                if (m < M && lane < 32) {
                    const int8_t* b = xq + (size_t)m * K + three + kSubK * u + 2 * lane;
                    uint32_t w[8];
                    pair_table(b[0], b[1], w);
                    store_table(lut + m * kTokenStride + lane * kSlot, w);
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int code = (int)((word >> (4 * i)) & 15u);
                const uint8_t* e = lut + (8 * q + i) * kSlot + 2 * code;
#pragma unroll
                for (int m = 0; m < MT; ++m) acc[m] += lds_i16(e + (m < M ? m : 0) * kTokenStride);
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        }
    }

    // Reduce: over the four q quarters (lanes r, r+16, r+32, r+48), then over waves.
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        int v = acc[m];
        v += __shfl_xor(v, 16, 64);
        v += __shfl_xor(v, 32, 64);
        acc[m] = v;
    }
    __syncthreads();   // every wave is done with its tables: reuse the LDS for the reduction
    int* red = reinterpret_cast<int*>(lds);
    if (lane < 16) {
#pragma unroll
        for (int m = 0; m < MT; ++m)
            if (m < M) red[(wave * 16 + m) * 16 + lane] = acc[m];
    }
    __syncthreads();
    if (wave != 0 || lane >= 16) return;
    const float beta = *w_scale;
    const int n = rg * kRowsPerGroup + r;
    for (int m = 0; m < M; ++m) {
        int s = 0;
        for (int w = 0; w < WAVES; ++w) s += red[(w * 16 + m) * 16 + lane];
        const float sc = beta / x_scale[m];
        y[(size_t)m * N + n] = (float)s * sc;
        if (acc_out) acc_out[(size_t)m * N + n] = s;
    }
}

// Standalone table precompute: the same tables, written to global memory for inspection.
__global__ __launch_bounds__(256) void elut_tables_kernel(const int8_t* __restrict__ xq, int M, int K,
                                                          int16_t* __restrict__ lut, int16_t* __restrict__ lut1) {
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    const int G = three / 3, P = (K - three) / 2;
    const size_t total = (size_t)M * (G + P);
    for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (size_t)gridDim.x * 256) {
        const int m = (int)(e / (size_t)(G + P));
        const int j = (int)(e - (size_t)m * (G + P));
        uint32_t w[8];
        uint8_t* dst;
        if (j < G) {
            const int8_t* a = xq + (size_t)m * K + 3 * j;
            triple_table(a[0], a[1], a[2], w);
            dst = reinterpret_cast<uint8_t*>(lut + ((size_t)m * G + j) * 16);
        } else {
            const int p = j - G;
            const int8_t* b = xq + (size_t)m * K + three + 2 * p;
            pair_table(b[0], b[1], w);
            dst = reinterpret_cast<uint8_t*>(lut1 + ((size_t)m * P + p) * 16);
        }
        store_table(dst, w);
    }
}

}  // namespace

int tl2_elut_waves(int M) {
    // Each wave holds M * kTokenStride bytes of tables; stay within 64 KiB per work group.
    int w = 16;
    while (w > 1 && (size_t)w * M * kTokenStride > 65536) w >>= 1;
    return w;
}

size_t tl2_elut_lds_bytes(int M) {
    const size_t tables = (size_t)tl2_elut_waves(M) * M * kTokenStride;
    const size_t red = (size_t)tl2_elut_waves(M) * 16 * 16 * sizeof(int);
    return tables > red ? tables : red;
}

template <int MT>
hipError_t launch_elut_mt(const uint8_t* pk, const float* w_scale, const int8_t* xq, const float* x_scale, int M,
                          int N, int K, float* y, int32_t* acc, hipStream_t stream) {
    const unsigned grid = (unsigned)(N / kRowsPerGroup);
    const size_t lds = tl2_elut_lds_bytes(M);
    switch (tl2_elut_waves(M)) {
        case 16:
            hipLaunchKernelGGL((tl2_elut_decode_kernel<16, MT>), dim3(grid), dim3(1024), lds, stream, pk, w_scale, xq,
                               x_scale, M, N, K, y, acc);
            break;
        case 8:
            hipLaunchKernelGGL((tl2_elut_decode_kernel<8, MT>), dim3(grid), dim3(512), lds, stream, pk, w_scale, xq,
                               x_scale, M, N, K, y, acc);
            break;
        case 4:
            hipLaunchKernelGGL((tl2_elut_decode_kernel<4, MT>), dim3(grid), dim3(256), lds, stream, pk, w_scale, xq,
                               x_scale, M, N, K, y, acc);
            break;
        case 2:
            hipLaunchKernelGGL((tl2_elut_decode_kernel<2, MT>), dim3(grid), dim3(128), lds, stream, pk, w_scale, xq,
                               x_scale, M, N, K, y, acc);
            break;
        default:
            hipLaunchKernelGGL((tl2_elut_decode_kernel<1, MT>), dim3(grid), dim3(64), lds, stream, pk, w_scale, xq,
                               x_scale, M, N, K, y, acc);
            break;
    }
    return hipGetLastError();
}

hipError_t launch_tl2_elut_decode(const void* packed, const float* w_scale, const int8_t* xq, const float* x_scale,
                                  int M, int N, int K, float* y, int32_t* acc, hipStream_t stream) {
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    if (M <= 1) return launch_elut_mt<1>(pk, w_scale, xq, x_scale, M, N, K, y, acc, stream);
    if (M <= 2) return launch_elut_mt<2>(pk, w_scale, xq, x_scale, M, N, K, y, acc, stream);
    if (M <= 4) return launch_elut_mt<4>(pk, w_scale, xq, x_scale, M, N, K, y, acc, stream);
    return launch_elut_mt<8>(pk, w_scale, xq, x_scale, M, N, K, y, acc, stream);
}

hipError_t launch_elut_tables(const int8_t* xq, int M, int K, int16_t* lut, int16_t* lut1, hipStream_t stream) {
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    const size_t total = (size_t)M * (three / 3 + (K - three) / 2);
    const unsigned grid = (unsigned)std::min<size_t>(4096, (total + 255) / 256);
    hipLaunchKernelGGL(elut_tables_kernel, dim3(grid > 0 ? grid : 1), dim3(256), 0, stream, xq, M, K, lut, lut1);
    return hipGetLastError();
}

}  // namespace bitnet
