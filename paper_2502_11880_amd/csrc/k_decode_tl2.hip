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
// Three kernels:
//   tl2_elut_decode_kernel   one work group per 16-row group; each wave takes every WAVES-th 384-k block, builds
//                            the tables of that block's 128 triples for up to 8 tokens in its own LDS slice and
//                            looks up its 16 rows x 128 triples (slices of different lane quarters skewed by 32 bytes
//                            so the quarters read disjoint banks); waves reduce through LDS.
//   tl2_stream_kernel        one token: persistent work groups build the tables of the whole row once and walk
//                            row groups (the table-lookup route where the tables fit in LDS).
//   tl2_mfma_decode_kernel   no activation tables: the packed triples are expanded to int8 weights through two
//                            small constant tables and multiplied on int8 MFMA, shared by up to 16 tokens.
#include "bitnet_internal.hpp"

#include <algorithm>
#include <type_traits>

namespace bitnet {
namespace {

constexpr int kSlot = 32;                                   // bytes per triple (or pair) table
constexpr int kTokenStride = (kTl2BlockK / 3 + 4) * kSlot;  // 128 triples + 4 skew slots per token
constexpr int kElutLdsBudget = 144 * 1024;                  // tables of a table-lookup work group
// Tokens whose TL2 tables a wave holds at once (16 waves x 2 x 4.1 KiB fit the budget).
constexpr int tl2_elut_chunk(int mt) { return mt < 2 ? mt : 2; }

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

// Lossy tables (TL2_0, TL1_0; Sec. 3.2.1): the smallest s >= 0 with max_abs <= 127 * 2^s, and an entry divided by
// 2^s and rounded half to even (the product by 2^-s is exact in fp32, rintf rounds ties to even).
__device__ __forceinline__ int lossy_shift_of(int max_abs) {
    int s = 0;
    while (max_abs > (127 << s)) ++s;
    return s;
}
__device__ __forceinline__ int lossy_q(int e, int s) {
    return s == 0 ? e : (int)rintf((float)e * __int_as_float((127 - s) << 23));
}
// The words of a table with every int16 entry quantised.
__device__ __forceinline__ void quantize_words(uint32_t w[8], int s) {
    if (s == 0) return;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int lo = (int)(int16_t)(w[i] & 0xFFFFu), hi = (int)(int16_t)(w[i] >> 16);
        w[i] = pack16(lossy_q(lo, s), lossy_q(hi, s));
    }
}
// Largest |entry| over the wave's tables of one token (each lane passes the largest of its own).
__device__ __forceinline__ int wave_max_int(int v) {
    return (int)wave_max_all((float)v);
}

// The int8 code of one activation (the quantiser's rounding: half to even, clamped to [-128, 127]).
__device__ __forceinline__ int code_of(float v, float s) {
    return (int)fminf(fmaxf(rintf(v * s), -128.0f), 127.0f);
}

// One token quantised inside a table-lookup launch (QX): the row's scale from its absmax (every work group reads the
// whole fp32 row, L2-resident after the first), the quantiser's formula.
template <int WAVES>
__device__ __forceinline__ float row_scale(const float* __restrict__ x, int K, float* red) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float4* x4 = reinterpret_cast<const float4*>(x);
    float amax = 0.0f;
    for (int i = tid; i < K / 4; i += 64 * WAVES) {
        const float4 v = x4[i];
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w))));
    }
    amax = wave_max_all(amax);
    if (lane == 0) red[wave] = amax;
    __syncthreads();
    amax = red[0];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) amax = fmaxf(amax, red[w]);
    return 127.0f / fmaxf(amax, 1e-5f);
}

// Work group 0 of a QX launch also writes the row's scale and code sum (its codes it stores as it makes them).
template <int WAVES>
__device__ __forceinline__ void write_row_sum(int csum, float sx, int* red, float* s_out, int32_t* rs_out) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    csum = wave_sum_all(csum);
    __syncthreads();
    if (lane == 0) red[wave] = csum;
    __syncthreads();
    if (tid == 0) {
        int tot = 0;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) tot += red[w];
        rs_out[0] = tot;
        s_out[0] = sx;
    }
}

// One work group per 16-row group of the launch's weights (rows of a fused group concatenated; the group's weight
// is found by a scalar compare chain).  LOSSY (TL2_0, Sec. 3.2.1): each token's tables of a block (128 triples, or
// the 32 pairs of a TL1 unit) are quantised to int8 with the block's power-of-two scale before the lookups, and the
// block's sum is scaled back.  QX (one token): the work group quantises the fp32 row itself and work group 0 writes
// the codes, the scale and their sum, as the quantiser would.
template <int WAVES, int MT, bool LOSSY, bool QX>
__global__ __launch_bounds__(64 * WAVES) void tl2_elut_decode_kernel(
    FusedLinears L, const float* __restrict__ x, const int8_t* __restrict__ xq, const float* __restrict__ x_scale,
    int M, int K, int8_t* __restrict__ xq_out, float* __restrict__ s_out, int32_t* __restrict__ rs_out) {
    extern __shared__ __align__(16) uint8_t lds[];
    __shared__ float redf[WAVES];
    __shared__ int redi[WAVES];
    static_assert(!QX || MT == 1, "the fused quantiser takes one token");
    constexpr int TC = tl2_elut_chunk(MT);      // tokens whose tables share LDS at a time
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int q = lane >> 4, r = lane & 15;
    int li, rg;
    locate(L, xcd_logical_id(blockIdx.x, gridDim.x), li, rg);
    const int N = pick(L.N, li);
    const uint8_t* packed = pick(L.packed, li);
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    const int nblk = three / kTl2BlockK;
    const int units = (K - three) / kSubK;
    const bool qw = QX && blockIdx.x == 0;      // this work group writes the codes
    const float sx = QX ? row_scale<WAVES>(x, K, redf) : 1.0f;
    int csum = 0;
    const uint8_t* idx_plane = packed;
    const uint8_t* sign_plane = packed + (size_t)N * (three / 6);
    const uint8_t* tail_plane = sign_plane + (size_t)N * (three / 24);
    uint8_t* lut = lds + (size_t)wave * TC * kTokenStride;

    int acc[MT];                                 // MT >= M tokens; loops run to MT with uniform guards
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = 0;

    for (int blk = wave; blk < nblk; blk += WAVES) {
        const size_t tile = (size_t)rg * nblk + blk;
        const v4u iw = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(idx_plane + tile * 1024 + 16 * lane));
        const uint32_t sw = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(sign_plane + tile * 256 + 4 * lane));
        const int nneg = __popc(sw);
        // tokens in chunks of TC: the chunk's tables of this block's 128 triples (lane builds triples lane and
        // lane + 64), then its lookups
#pragma unroll
        for (int c = 0; c < MT; c += TC) {
            if (c >= M) break;
            int shift[TC];
#pragma unroll
            for (int j = 0; j < TC; ++j) shift[j] = 0;
#pragma unroll
            for (int j = 0; j < TC; ++j) {
                const int m = c + j;
                if (m >= M) break;
                // the codes of triples lane and lane + 64
                int cd[2][3];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int g = lane + 64 * h;
                    const size_t k = (size_t)blk * kTl2BlockK + 3 * g;
#pragma unroll
                    for (int e = 0; e < 3; ++e) {
                        if constexpr (QX) {
                            cd[h][e] = code_of(x[k + e], sx);
                            if (qw) {
                                xq_out[k + e] = (int8_t)cd[h][e];
                                csum += cd[h][e];
                            }
                        } else {
                            cd[h][e] = xq[(size_t)m * K + k + e];
                        }
                    }
                }
                if constexpr (LOSSY) {
                    // the block's largest |entry| is the largest |a0| + |a1| + |a2| of its triples
                    int mx = 0;
#pragma unroll
                    for (int h = 0; h < 2; ++h) mx = max(mx, abs(cd[h][0]) + abs(cd[h][1]) + abs(cd[h][2]));
                    shift[j] = lossy_shift_of(wave_max_int(mx));
                }
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int g = lane + 64 * h;
                    uint32_t w[8];
                    triple_table(cd[h][0], cd[h][1], cd[h][2], w);
                    if constexpr (LOSSY) quantize_words(w, shift[j]);
                    store_table(lut + j * kTokenStride + skewed_slot(g) * kSlot, w);
                }
            }
            wave_lds_handoff();
            // Lookups without branches: tokens past M read the chunk's first tables and are never stored, so all
            // 32 x TC reads of a lane can be in flight together (a guarded read per triple waits for each one).
            const uint8_t* base = lut + skewed_slot(32 * q) * kSlot;
            int bsum[TC];
#pragma unroll
            for (int j = 0; j < TC; ++j) bsum[j] = 0;
#pragma unroll
            for (int i = 0; i < 32; ++i) {
                const uint32_t word = i < 8 ? iw.x : i < 16 ? iw.y : i < 24 ? iw.z : iw.w;
                const int idx = (int)((word >> (4 * (i & 7))) & 15u);
                const int msk = -(int)((sw >> i) & 1u);
                const uint8_t* e = base + i * kSlot + 2 * idx;
#pragma unroll
                for (int j = 0; j < TC; ++j) bsum[j] += lds_i16(e + (c + j < M ? j : 0) * kTokenStride) ^ msk;
            }
#pragma unroll
            for (int j = 0; j < TC; ++j)
                if (c + j < MT) acc[c + j] += (bsum[j] + nneg) << shift[j];
            wave_lds_handoff();
        }
    }

    // TL1 tail (K mod 384 weights): handled by the wave after the last TL2 block.
    if (units > 0 && wave == nblk % WAVES) {
        for (int u = 0; u < units; ++u) {
            const uint32_t word = *reinterpret_cast<const uint32_t*>(
                tail_plane + ((size_t)rg * 64 * units + (size_t)lane * units + u) * 4);
#pragma unroll
            for (int c = 0; c < MT; c += TC) {
                if (c >= M) break;
                // pair tables of this unit's 32 pairs (k = three + 64u + 2p), lanes 0..31
                int shift[TC];
#pragma unroll
                for (int j = 0; j < TC; ++j) shift[j] = 0;
#pragma unroll
                for (int j = 0; j < TC; ++j) {
                    const int m = c + j;
                    if (m >= M) break;
                    const size_t k = (size_t)three + kSubK * u + 2 * (lane & 31);
                    int b0, b1;
                    if constexpr (QX) {
                        b0 = code_of(x[k], sx);
                        b1 = code_of(x[k + 1], sx);
                        if (qw && lane < 32) {
                            xq_out[k] = (int8_t)b0;
                            xq_out[k + 1] = (int8_t)b1;
                            csum += b0 + b1;
                        }
                    } else {
                        b0 = xq[(size_t)m * K + k];
                        b1 = xq[(size_t)m * K + k + 1];
                    }
                    if constexpr (LOSSY)
                        shift[j] = lossy_shift_of(wave_max_int(lane < 32 ? abs(b0) + abs(b1) : 0));
                    if (lane < 32) {
                        uint32_t w[8];
                        pair_table(b0, b1, w);
                        if constexpr (LOSSY) quantize_words(w, shift[j]);
                        store_table(lut + j * kTokenStride + lane * kSlot, w);
                    }
                }
                wave_lds_handoff();
                int usum[TC];
#pragma unroll
                for (int j = 0; j < TC; ++j) usum[j] = 0;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int code = (int)((word >> (4 * i)) & 15u);
                    const uint8_t* e = lut + (8 * q + i) * kSlot + 2 * code;
#pragma unroll
                    for (int j = 0; j < TC; ++j) usum[j] += lds_i16(e + (c + j < M ? j : 0) * kTokenStride);
                }
#pragma unroll
                for (int j = 0; j < TC; ++j)
                    if (c + j < MT) acc[c + j] += usum[j] << shift[j];
                wave_lds_handoff();
            }
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
    if constexpr (QX) {
        if (qw) write_row_sum<WAVES>(csum, sx, redi, s_out, rs_out);
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
    const float beta = *pick(L.w_scale, li);
    float* y = pick(L.y, li);
    int32_t* acc_out = pick(L.acc, li);
    const int n = rg * kRowsPerGroup + r;
    for (int m = 0; m < M; ++m) {
        int s = 0;
        for (int w = 0; w < WAVES; ++w) s += red[(w * 16 + m) * 16 + lane];
        const float sc = beta / (QX ? sx : x_scale[m]);
        y[(size_t)m * N + n] = (float)s * sc;
        if (acc_out) acc_out[(size_t)m * N + n] = s;
    }
}

// The TL1 layout by table lookup (Algorithm TL1; Table 5), one work group per 16-row group: wave w takes the 256-k
// blocks w, w + WAVES, ... (four 64-k units each, the last block possibly fewer); lane l builds the 9-entry tables
// of pair l % 32 of units l / 32 and 2 + l / 32, for a chunk of up to two tokens at a time, and lane (r, q) looks
// up the 8 pairs of each of its block's words (row r, k = 64 j + 16 q .. + 15 of unit j).  LOSSY (TL1_0, Sec. 3.2.1):
// each token's tables of a unit are quantised to int8 with the unit's power-of-two scale and the unit's sum is
// scaled back.  Fused weight groups and QX as for the TL2 kernel.
constexpr int kTl1BlockStride = 128 * kSlot;                 // the 128 pair tables of a 256-k block per token

// Largest value of each half-wave (lanes 0..31 and 32..63) of v, as scalars: DPP maxima inside each row of 16 lanes,
// then the four row results read from lanes 0, 16, 32 and 48.
__device__ __forceinline__ void half_wave_max(int v, int& lo, int& hi) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v = max(v, dpp_row_step(v, i));
    lo = max(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 16));
    hi = max(__builtin_amdgcn_readlane(v, 32), __builtin_amdgcn_readlane(v, 48));
}

template <int WAVES, int MT, bool LOSSY, bool QX>
__global__ __launch_bounds__(64 * WAVES) void tl1_elut_decode_kernel(
    FusedLinears L, const float* __restrict__ x, const int8_t* __restrict__ xq, const float* __restrict__ x_scale,
    int M, int K, int8_t* __restrict__ xq_out, float* __restrict__ s_out, int32_t* __restrict__ rs_out) {
    extern __shared__ __align__(16) uint8_t lds[];
    __shared__ float redf[WAVES];
    __shared__ int redi[WAVES];
    static_assert(!QX || MT == 1, "the fused quantiser takes one token");
    constexpr int TC = tl2_elut_chunk(MT);      // tokens whose tables share LDS at a time
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int q = lane >> 4, r = lane & 15;
    const int pr = lane & 31, hh = lane >> 5;  // this lane builds pair pr of units hh and 2 + hh
    int li, rg;
    locate(L, xcd_logical_id(blockIdx.x, gridDim.x), li, rg);
    const int N = pick(L.N, li);
    const uint8_t* packed = pick(L.packed, li);
    const bool qw = QX && blockIdx.x == 0;      // this work group writes the codes
    const float sx = QX ? row_scale<WAVES>(x, K, redf) : 1.0f;
    int csum = 0;
    const int nsub = K / kSubK;
    const int nkb = (nsub + 3) / 4;
    const uint8_t* rgbase = packed + (size_t)rg * 4 * K;
    uint8_t* lut = lds + (size_t)wave * TC * kTl1BlockStride;

    int acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = 0;

    for (int sb = wave; sb < nkb; sb += WAVES) {
        const int T = min(4, nsub - 4 * sb);   // units of this block
        // the lane's word of unit j: word j of its 4 T bytes in the I2_S tiling (units past T repeat a real word)
        uint32_t word[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            word[j] = *reinterpret_cast<const uint32_t*>(rgbase + (size_t)sb * 1024 + 4 * T * lane + 4 * min(j, T - 1));
        const bool ok0 = hh < T, ok1 = 2 + hh < T;
        const int u0 = min(hh, T - 1), u1 = min(2 + hh, T - 1);
#pragma unroll
        for (int c = 0; c < MT; c += TC) {
            if (c >= M) break;
            int sh[TC][4];
#pragma unroll
            for (int jj = 0; jj < TC; ++jj)
#pragma unroll
                for (int j = 0; j < 4; ++j) sh[jj][j] = 0;
#pragma unroll
            for (int jj = 0; jj < TC; ++jj) {
                const int m = c + jj;
                if (m >= M) break;
                const size_t kb0 = (size_t)sb * kI2sBlockK + 2 * pr;
                int a0, a1, b0, b1;
                if constexpr (QX) {
                    a0 = code_of(x[kb0 + kSubK * u0], sx);
                    a1 = code_of(x[kb0 + kSubK * u0 + 1], sx);
                    b0 = code_of(x[kb0 + kSubK * u1], sx);
                    b1 = code_of(x[kb0 + kSubK * u1 + 1], sx);
                    if (qw) {
                        if (ok0) {
                            xq_out[kb0 + kSubK * u0] = (int8_t)a0;
                            xq_out[kb0 + kSubK * u0 + 1] = (int8_t)a1;
                            csum += a0 + a1;
                        }
                        if (ok1) {
                            xq_out[kb0 + kSubK * u1] = (int8_t)b0;
                            xq_out[kb0 + kSubK * u1 + 1] = (int8_t)b1;
                            csum += b0 + b1;
                        }
                    }
                } else {
                    const int8_t* xb = xq + (size_t)m * K + kb0;
                    a0 = xb[kSubK * u0];
                    a1 = xb[kSubK * u0 + 1];
                    b0 = xb[kSubK * u1];
                    b1 = xb[kSubK * u1 + 1];
                }
                if constexpr (LOSSY) {
                    int lo0, hi0, lo1, hi1;
                    half_wave_max(ok0 ? abs(a0) + abs(a1) : 0, lo0, hi0);
                    half_wave_max(ok1 ? abs(b0) + abs(b1) : 0, lo1, hi1);
                    sh[jj][0] = lossy_shift_of(lo0);
                    sh[jj][1] = lossy_shift_of(hi0);
                    sh[jj][2] = lossy_shift_of(lo1);
                    sh[jj][3] = lossy_shift_of(hi1);
                }
                uint32_t w[8];
                uint8_t* tj = lut + jj * kTl1BlockStride;
                if (ok0) {
                    pair_table(a0, a1, w);
                    if constexpr (LOSSY) quantize_words(w, hh ? sh[jj][1] : sh[jj][0]);
                    store_table(tj + (32 * hh + pr) * kSlot, w);
                }
                if (ok1) {
                    pair_table(b0, b1, w);
                    if constexpr (LOSSY) quantize_words(w, hh ? sh[jj][3] : sh[jj][2]);
                    store_table(tj + (64 + 32 * hh + pr) * kSlot, w);
                }
            }
            wave_lds_handoff();
            // lookups: tokens past M read the chunk's first tables and are never stored
            int usum[TC][4];
#pragma unroll
            for (int jj = 0; jj < TC; ++jj)
#pragma unroll
                for (int j = 0; j < 4; ++j) usum[jj][j] = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (j >= T) break;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    // pair i of the word: byte i % 4, low nibble for i < 4; it is pair 8 q + i of unit j
                    const int code = (int)((word[j] >> (8 * (i & 3) + 4 * (i >> 2))) & 15u);
                    const uint8_t* e = lut + (32 * j + 8 * q + i) * kSlot + 2 * code;
#pragma unroll
                    for (int jj = 0; jj < TC; ++jj)
                        usum[jj][j] += lds_i16(e + (c + jj < M ? jj : 0) * kTl1BlockStride);
                }
            }
#pragma unroll
            for (int jj = 0; jj < TC; ++jj)
                if (c + jj < MT)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[c + jj] += usum[jj][j] << sh[jj][j];
            wave_lds_handoff();
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
    if constexpr (QX) {
        if (qw) write_row_sum<WAVES>(csum, sx, redi, s_out, rs_out);
    }
    __syncthreads();
    int* red = reinterpret_cast<int*>(lds);
    if (lane < 16) {
#pragma unroll
        for (int m = 0; m < MT; ++m)
            if (m < M) red[(wave * 16 + m) * 16 + lane] = acc[m];
    }
    __syncthreads();
    if (wave != 0 || lane >= 16) return;
    const float beta = *pick(L.w_scale, li);
    float* y = pick(L.y, li);
    int32_t* acc_out = pick(L.acc, li);
    const int n = rg * kRowsPerGroup + r;
    for (int m = 0; m < M; ++m) {
        int s = 0;
        for (int w = 0; w < WAVES; ++w) s += red[(w * 16 + m) * 16 + lane];
        y[(size_t)m * N + n] = (float)s * (beta / (QX ? sx : x_scale[m]));
        if (acc_out) acc_out[(size_t)m * N + n] = s;
    }
}

// One token, streaming (Algorithm TL2 with the table build amortised over every row the work group visits).
// Each persistent work group quantises the token row once (Sec. 2.1; or reads the codes when they are given), then
// every wave builds the tables of its own 384-k blocks once: 14 int16 sums in a 28-byte slot per triple, 132
// slots per block (a one-slot skew after every 32 triples puts the four lane quarters on disjoint banks), and the
// wave holding the TL1 tail builds its pair tables.  The work group then walks the row groups g = blockIdx.x +
// j gridDim.x of all the launch's weights: the next row group's index and sign words are loaded while the current
// one is looked up, and one barrier per row group reduces the waves' sums (double-buffered) for the epilogue.
constexpr int kSlot28 = 28;                                  // 14 int16 per triple table
constexpr int kBlockBytes28 = (kTl2BlockK / 3 + 4) * kSlot28;
constexpr int kMaxUnits = kTl2BlockK / kSubK - 1;            // TL1 tail: at most 5 units of 64 k

__device__ __forceinline__ void store_words(uint8_t* slot, const uint32_t* w, int n) {
    for (int i = 0; i < n; ++i) reinterpret_cast<uint32_t*>(slot)[i] = w[i];
}

template <int WAVES, int U, int XV, bool QUANT, bool LOSSY>
__global__ __launch_bounds__(64 * WAVES) void tl2_stream_kernel(FusedLinears L, const float* __restrict__ x, int K,
                                                                int8_t* __restrict__ xq, float* __restrict__ x_scale,
                                                                int32_t* __restrict__ x_rowsum) {
    extern __shared__ __align__(16) uint8_t lds[];    // codes | block tables | pair tables
    __shared__ int part[2][WAVES][16];
    __shared__ float redf[WAVES];
    __shared__ int redi[WAVES];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q = lane >> 4;
    const int G = gridDim.x, bid = blockIdx.x;
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    const int nblk = three / kTl2BlockK;
    const int units = (K - three) / kSubK;
    const int tail_wave = nblk % WAVES;                        // a wave with the fewest blocks
    uint8_t* codes = lds;
    uint8_t* tables = lds + ((K + 15) & ~15);
    uint8_t* pairs = tables + (size_t)nblk * kBlockBytes28;
    const int S = (L.total - bid + G - 1) / G;                 // row groups of this work group (grid <= total)

    // the loads of row group step st (all unconditional: a conditional load shape makes the compiler wait for
    // every load in flight where the paths join); blocks past nblk and tail units past `units` repeat real ones
    auto issue = [&](v4u (&iw)[U], uint32_t (&sw)[U], uint32_t (&tw)[kMaxUnits], float& bw, int st) {
        int li, rg;
        locate(L, bid + st * G, li, rg);
        const size_t Nl = (size_t)pick(L.N, li);
        const uint8_t* idx_plane = pick(L.packed, li);
        const uint8_t* sign_plane = idx_plane + Nl * (three / 6);
        const uint8_t* tail_plane = sign_plane + Nl * (three / 24);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t tile = (size_t)rg * nblk + min(wave + WAVES * u, nblk - 1);
            iw[u] = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(idx_plane + tile * 1024 + 16 * lane));
            sw[u] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(sign_plane + tile * 256 + 4 * lane));
        }
        // without a tail the words are read from the start of the index plane instead (never used)
        const int um = units > 0 ? units : 1;
        const uint8_t* tail_base = units > 0 ? tail_plane : idx_plane;
        const size_t tail_row = units > 0 ? ((size_t)rg * 64 * um + (size_t)lane * um) : 0;
#pragma unroll
        for (int t = 0; t < kMaxUnits; ++t)
            tw[t] = *reinterpret_cast<const uint32_t*>(tail_base + (tail_row + (units > 0 ? min(t, um - 1) : 0)) * 4);
        bw = *pick(L.w_scale, li);
    };

    auto run = [&](auto multi) {
        constexpr bool kMulti = decltype(multi)::value;
        // 1. the activation row, the first row groups' weights, then the quantisation (or the given codes)
        const float4* x4 = reinterpret_cast<const float4*>(x);
        const int K4 = K >> 2;
        float4 xv[XV];
        if (QUANT) {
#pragma unroll
            for (int i = 0; i < XV; ++i) {
                const int e = tid + i * 64 * WAVES;
                const float4 v = x4[e < K4 ? e : K4 - 1];
                xv[i] = e < K4 ? v : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            }
        }
        v4u iwa[U], iwb[U];
        uint32_t swa[U], swb[U], twa[kMaxUnits], twb[kMaxUnits];
        float ba = 0.0f, bb = 0.0f;
        issue(iwa, swa, twa, ba, 0);
        if constexpr (kMulti) issue(iwb, swb, twb, bb, 1);
        __builtin_amdgcn_sched_barrier(0);
        float sx;
        if (QUANT) {
            float amax = 0.0f;
#pragma unroll
            for (int i = 0; i < XV; ++i)
                amax = fmaxf(amax, fmaxf(fmaxf(fabsf(xv[i].x), fabsf(xv[i].y)), fmaxf(fabsf(xv[i].z), fabsf(xv[i].w))));
            amax = wave_max_all(amax);
            if (lane == 0) redf[wave] = amax;
            __syncthreads();
            amax = redf[0];
#pragma unroll
            for (int w = 1; w < WAVES; ++w) amax = fmaxf(amax, redf[w]);
            sx = 127.0f / fmaxf(amax, 1e-5f);
            int sum = 0;
#pragma unroll
            for (int i = 0; i < XV; ++i) {
                const int e = tid + i * 64 * WAVES;
                if (e < K4) {
                    const uint32_t c = quant4(xv[i], sx);
                    sum = byte_sum4(c, sum);
                    reinterpret_cast<uint32_t*>(codes)[e] = c;
                    if (bid == 0) reinterpret_cast<uint32_t*>(xq)[e] = c;
                }
            }
            sum = wave_sum_all(sum);
            if (lane == 0) redi[wave] = sum;
        } else {
            for (int e = tid; e < K4; e += 64 * WAVES)
                reinterpret_cast<uint32_t*>(codes)[e] = reinterpret_cast<const uint32_t*>(xq)[e];
            sx = x_scale[0];
        }
        __syncthreads();                                   // every code (and every wave's code sum) is in LDS
        if (QUANT && bid == 0 && tid == 0) {
            int tot = 0;
            for (int w = 0; w < WAVES; ++w) tot += redi[w];
            x_scale[0] = sx;
            x_rowsum[0] = tot;
        }

        // 2. this wave's tables, once: lane builds triples lane and lane + 64 of each of its blocks.  LOSSY (TL2_0,
        //    Sec. 3.2.1): each block's tables (and each tail unit's pair tables) quantised to int8 with the block's
        //    power-of-two scale; the wave that builds a block is the one that looks it up, so the shifts stay in its
        //    registers
        int bshift[U], tshift[kMaxUnits];
#pragma unroll
        for (int u = 0; u < U; ++u) bshift[u] = 0;
#pragma unroll
        for (int t = 0; t < kMaxUnits; ++t) tshift[t] = 0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int blk = wave + WAVES * u;
            if (blk < nblk) {
                const int8_t* a0 = reinterpret_cast<const int8_t*>(codes) + blk * kTl2BlockK + 3 * lane;
                if constexpr (LOSSY) {
                    // the block's largest |entry|: the largest |a0| + |a1| + |a2| of its triples
                    int mx = 0;
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const int8_t* a = a0 + 3 * 64 * h;
                        mx = max(mx, abs((int)a[0]) + abs((int)a[1]) + abs((int)a[2]));
                    }
                    bshift[u] = lossy_shift_of(wave_max_int(mx));
                }
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int g = lane + 64 * h;
                    const int8_t* a = a0 + 3 * 64 * h;
                    uint32_t w[8];
                    triple_table(a[0], a[1], a[2], w);
                    if constexpr (LOSSY) quantize_words(w, bshift[u]);
                    store_words(tables + blk * kBlockBytes28 + skewed_slot(g) * kSlot28, w, 7);
                }
            }
        }
        if (wave == tail_wave) {
#pragma unroll
            for (int t = 0; t < kMaxUnits; ++t) {
                if (t < units) {
                    const int8_t* b = reinterpret_cast<const int8_t*>(codes) + three + kSubK * t + 2 * (lane & 31);
                    if constexpr (LOSSY)
                        tshift[t] = lossy_shift_of(wave_max_int(lane < 32 ? abs((int)b[0]) + abs((int)b[1]) : 0));
                    if (lane < 32) {
                        uint32_t w[8];
                        pair_table(b[0], b[1], w);
                        if constexpr (LOSSY) quantize_words(w, tshift[t]);
                        store_words(pairs + (t * 32 + lane) * kSlot28, w, 5);
                    }
                }
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");

        // 3. the stream
        int par = 0;
        auto compute = [&](const v4u (&iw)[U], const uint32_t (&sw)[U], const uint32_t (&tw)[kMaxUnits], float bw,
                           int st) {
            int acc = 0;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int blk = wave + WAVES * u;
                if (blk < nblk) {
                    const uint8_t* base = tables + blk * kBlockBytes28 + skewed_slot(32 * q) * kSlot28;
                    int bsum = 0;
#pragma unroll
                    for (int i = 0; i < 32; ++i) {
                        const uint32_t word = i < 8 ? iw[u].x : i < 16 ? iw[u].y : i < 24 ? iw[u].z : iw[u].w;
                        const int idx = (int)((word >> (4 * (i & 7))) & 15u);
                        const int msk = -(int)((sw[u] >> i) & 1u);
                        bsum += lds_i16(base + i * kSlot28 + 2 * idx) ^ msk;
                    }
                    bsum += __popc(sw[u]);
                    acc += LOSSY ? bsum << bshift[u] : bsum;
                }
            }
            if (wave == tail_wave) {
#pragma unroll
                for (int t = 0; t < kMaxUnits; ++t) {
                    if (t < units) {
                        int usum = 0;
#pragma unroll
                        for (int i = 0; i < 8; ++i) {
                            const int code = (int)((tw[t] >> (4 * i)) & 15u);
                            usum += lds_i16(pairs + (t * 32 + 8 * q + i) * kSlot28 + 2 * code);
                        }
                        acc += LOSSY ? usum << tshift[t] : usum;
                    }
                }
            }
            acc += __shfl_xor(acc, 16, 64);
            acc += __shfl_xor(acc, 32, 64);
            if (lane < 16) part[par][wave][lane] = acc;
            __syncthreads();
            if (wave == 0 && lane < 16) {
                int v = 0;
#pragma unroll
                for (int w = 0; w < WAVES; ++w) v += part[par][w][lane];
                int li, rg;
                locate(L, bid + st * G, li, rg);
                const int n = rg * kRowsPerGroup + lane;
                pick(L.y, li)[n] = (float)v * (bw / sx);
                int32_t* acc_out = pick(L.acc, li);
                if (acc_out) acc_out[n] = v;
            }
            par ^= 1;
        };
        if constexpr (!kMulti) {
            compute(iwa, swa, twa, ba, 0);
            return;
        }
        int st = 0;
        for (; st + 3 < S; st += 2) {
            compute(iwa, swa, twa, ba, st);
            issue(iwa, swa, twa, ba, st + 2);
            compute(iwb, swb, twb, bb, st + 1);
            issue(iwb, swb, twb, bb, st + 3);
        }
        if (st + 2 < S) {
            compute(iwa, swa, twa, ba, st);
            issue(iwa, swa, twa, ba, st + 2);
            compute(iwb, swb, twb, bb, st + 1);
            compute(iwa, swa, twa, ba, st + 2);
        } else {
            compute(iwa, swa, twa, ba, st);
            compute(iwb, swb, twb, bb, st + 1);
        }
    };
    if (S == 1) run(std::false_type{});
    else run(std::true_type{});
}

// One token, TL1_0 (lossy TL1, Table 1; Sec. 3.2.1), persistent: each work group quantises the row (or copies the
// given codes), builds the pair tables (Table 5, Algorithm TL1) of the whole row once, each unit's tables quantised
// to int8 with the unit's power-of-two scale, and then walks the row groups g = blockIdx.x, blockIdx.x + gridDim.x,
// ... of all the launch's weights with the next row group's words in flight.  Wave w builds and reads the tables of
// blocks w, w + WAVES, ... (256 k each: 4 units of 32 pairs), so the unit shifts stay in its registers.
constexpr int kSlot20 = 20;                                  // 10 int16 per pair table (9 used)
constexpr int kTl1BlockBytes20 = 128 * kSlot20;               // the 128 pair tables of a 256-k block

template <int WAVES, int U, int XV, bool QUANT>
__global__ __launch_bounds__(64 * WAVES) void tl1_lossy_stream_kernel(FusedLinears L, const float* __restrict__ x,
                                                                      int K, int8_t* __restrict__ xq,
                                                                      float* __restrict__ x_scale,
                                                                      int32_t* __restrict__ x_rowsum) {
    extern __shared__ __align__(16) uint8_t lds[];    // codes | pair tables
    __shared__ int part[2][WAVES][16];
    __shared__ float redf[WAVES];
    __shared__ int redi[WAVES];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q = lane >> 4;
    const int pr = lane & 31, hh = lane >> 5;                  // this lane builds pair pr of units hh and 2 + hh
    const int G = gridDim.x, bid = blockIdx.x;
    const int nsub = K / kSubK;
    const int nkb = (nsub + 3) / 4;
    uint8_t* codes = lds;
    uint8_t* tables = lds + ((K + 15) & ~15);
    const int S = (L.total - bid + G - 1) / G;                 // row groups of this work group (grid <= total)

    // the loads of row group step st: word j of the lane's 4 T bytes of each of its blocks in the I2_S tiling (units
    // past T, and blocks past nkb, repeat real words; all unconditional)
    auto issue = [&](uint32_t (&wd)[U][4], float& bw, int st) {
        int li, rg;
        locate(L, bid + st * G, li, rg);
        const uint8_t* rgbase = pick(L.packed, li) + (size_t)rg * 4 * K;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int blk = min(wave + WAVES * u, nkb - 1);
            const int T = min(4, nsub - 4 * blk);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                wd[u][j] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(
                    rgbase + (size_t)blk * 1024 + 4 * T * lane + 4 * min(j, T - 1)));
        }
        bw = *pick(L.w_scale, li);
    };

    auto run = [&](auto multi) {
        constexpr bool kMulti = decltype(multi)::value;
        // 1. the activation row, the first row group's words, then the quantisation (or the given codes)
        const float4* x4 = reinterpret_cast<const float4*>(x);
        const int K4 = K >> 2;
        float4 xv[XV];
        if (QUANT) {
#pragma unroll
            for (int i = 0; i < XV; ++i) {
                const int e = tid + i * 64 * WAVES;
                const float4 v = x4[e < K4 ? e : K4 - 1];
                xv[i] = e < K4 ? v : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            }
        }
        uint32_t wa[U][4], wb[U][4];
        float ba = 0.0f, bb = 0.0f;
        issue(wa, ba, 0);
        __builtin_amdgcn_sched_barrier(0);
        float sx;
        if (QUANT) {
            float amax = 0.0f;
#pragma unroll
            for (int i = 0; i < XV; ++i)
                amax = fmaxf(amax, fmaxf(fmaxf(fabsf(xv[i].x), fabsf(xv[i].y)), fmaxf(fabsf(xv[i].z), fabsf(xv[i].w))));
            amax = wave_max_all(amax);
            if (lane == 0) redf[wave] = amax;
            __syncthreads();
            amax = redf[0];
#pragma unroll
            for (int w = 1; w < WAVES; ++w) amax = fmaxf(amax, redf[w]);
            sx = 127.0f / fmaxf(amax, 1e-5f);
            int sum = 0;
#pragma unroll
            for (int i = 0; i < XV; ++i) {
                const int e = tid + i * 64 * WAVES;
                if (e < K4) {
                    const uint32_t c = quant4(xv[i], sx);
                    sum = byte_sum4(c, sum);
                    reinterpret_cast<uint32_t*>(codes)[e] = c;
                    if (bid == 0) reinterpret_cast<uint32_t*>(xq)[e] = c;
                }
            }
            sum = wave_sum_all(sum);
            if (lane == 0) redi[wave] = sum;
        } else {
            for (int e = tid; e < K4; e += 64 * WAVES)
                reinterpret_cast<uint32_t*>(codes)[e] = reinterpret_cast<const uint32_t*>(xq)[e];
            sx = x_scale[0];
        }
        if constexpr (kMulti) issue(wb, bb, 1);
        __syncthreads();                                   // every code (and every wave's code sum) is in LDS
        if (QUANT && bid == 0 && tid == 0) {
            int tot = 0;
            for (int w = 0; w < WAVES; ++w) tot += redi[w];
            x_scale[0] = sx;
            x_rowsum[0] = tot;
        }

        // 2. this wave's tables, once, and the shift of each of their units
        int bsh[U][4];
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int j = 0; j < 4; ++j) bsh[u][j] = 0;
            const int blk = wave + WAVES * u;
            if (blk < nkb) {
                const int T = min(4, nsub - 4 * blk);
                const bool ok0 = hh < T, ok1 = 2 + hh < T;
                const int u0 = min(hh, T - 1), u1 = min(2 + hh, T - 1);
                const int8_t* cb = reinterpret_cast<const int8_t*>(codes) + blk * kI2sBlockK + 2 * pr;
                const int a0 = cb[kSubK * u0], a1 = cb[kSubK * u0 + 1];
                const int b0 = cb[kSubK * u1], b1 = cb[kSubK * u1 + 1];
                int lo0, hi0, lo1, hi1;
                half_wave_max(ok0 ? abs(a0) + abs(a1) : 0, lo0, hi0);
                half_wave_max(ok1 ? abs(b0) + abs(b1) : 0, lo1, hi1);
                bsh[u][0] = lossy_shift_of(lo0);
                bsh[u][1] = lossy_shift_of(hi0);
                bsh[u][2] = lossy_shift_of(lo1);
                bsh[u][3] = lossy_shift_of(hi1);
                uint8_t* tb = tables + (size_t)blk * kTl1BlockBytes20;
                uint32_t w[8];
                if (ok0) {
                    pair_table(a0, a1, w);
                    quantize_words(w, hh ? bsh[u][1] : bsh[u][0]);
                    store_words(tb + (32 * hh + pr) * kSlot20, w, 5);
                }
                if (ok1) {
                    pair_table(b0, b1, w);
                    quantize_words(w, hh ? bsh[u][3] : bsh[u][2]);
                    store_words(tb + (64 + 32 * hh + pr) * kSlot20, w, 5);
                }
            }
        }
        // the tables a lane wrote are read by the other lanes of its wave only
        wave_lds_handoff();

        // 3. the stream
        int par = 0;
        auto compute = [&](const uint32_t (&wd)[U][4], float bw, int st) {
            int acc = 0;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int blk = wave + WAVES * u;
                if (blk < nkb) {
                    const int T = min(4, nsub - 4 * blk);
                    const uint8_t* tb = tables + (size_t)blk * kTl1BlockBytes20;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if (j < T) {
                            int us = 0;
#pragma unroll
                            for (int i = 0; i < 8; ++i) {
                                // pair i of the word: byte i % 4, low nibble for i < 4; pair 8 q + i of unit j
                                const int code = (int)((wd[u][j] >> (8 * (i & 3) + 4 * (i >> 2))) & 15u);
                                us += lds_i16(tb + (32 * j + 8 * q + i) * kSlot20 + 2 * code);
                            }
                            acc += us << bsh[u][j];
                        }
                    }
                }
            }
            acc += __shfl_xor(acc, 16, 64);
            acc += __shfl_xor(acc, 32, 64);
            if (lane < 16) part[par][wave][lane] = acc;
            __syncthreads();
            if (wave == 0 && lane < 16) {
                int v = 0;
#pragma unroll
                for (int w = 0; w < WAVES; ++w) v += part[par][w][lane];
                int li, rg;
                locate(L, bid + st * G, li, rg);
                const int n = rg * kRowsPerGroup + lane;
                pick(L.y, li)[n] = (float)v * (bw / sx);
                int32_t* acc_out = pick(L.acc, li);
                if (acc_out) acc_out[n] = v;
            }
            par ^= 1;
        };
        if constexpr (!kMulti) {
            compute(wa, ba, 0);
            return;
        }
        int st = 0;
        for (; st + 3 < S; st += 2) {
            compute(wa, ba, st);
            issue(wa, ba, st + 2);
            compute(wb, bb, st + 1);
            issue(wb, bb, st + 3);
        }
        if (st + 2 < S) {
            compute(wa, ba, st);
            issue(wa, ba, st + 2);
            compute(wb, bb, st + 1);
            compute(wa, ba, st + 2);
        } else {
            compute(wa, ba, st);
            compute(wb, bb, st + 1);
        }
    };
    if (S == 1) run(std::false_type{});
    else run(std::true_type{});
}

// Several tokens (up to 16 per launch), TL2 on int8 MFMA.  Table lookups cost one LDS read per token and triple,
// so past one token the packed triples are instead expanded to int8 weights in registers and multiplied on
// v_mfma_i32_16x16x64_i8, the same contraction the I2_S kernels run; the expansion is shared by every token.
// Two small tables in LDS do the expansion (Eq. 5: a set sign bit negates all three weights of its triple):
//   - index table, 1024 entries of 8 bytes: a byte of the index plane (the 4-bit indices of two neighbouring
//     triples) and their two sign bits give the six weights, one signed byte each;
//   - pair table, 256 entries of 4 bytes: a byte of a TL1 tail word (two 4-bit pair codes, Table 5) gives
//     the four weights.
// Lane (q, r) holds triples 32q .. 32q+31 of row r of a 384-k block, that is k = 96q .. 96q+95 of the block in
// order; MFMA step s (0..5) takes the lane's weights 16s .. 16s+15, so its A operand is the tokens' codes at
// k = 96q + 16s.  (The contraction pairs A and B bytes by lane quarter and byte position, so any k order the two
// operands share gives the same sum.)  A tail unit's word holds k = 16q .. 16q+15 of its 64, in order.
// The weights are signed, so no code-sum correction is needed.
//
// Persistent work groups: each wave copies the codes of its own blocks (every token) into LDS and the group
// builds the two tables; then the group walks row groups g = blockIdx.x + j gridDim.x of all the launch's weights
// with the next row group's index, sign and tail words in flight, one barrier per row group for the reduction.
constexpr int kIdxTableBytes = 1024 * 8;
constexpr int kPairTableBytes = 256 * 4;
constexpr int kTl2MfmaTables = kIdxTableBytes + kPairTableBytes;
constexpr int kTl2MfmaMaxBlocks = 48;                         // 16 waves x 3 blocks

// Weight of balanced-ternary digit d (0 = leading) of a triple index 0..13 (index = 9 d0 + 3 d1 + d2); 0 for the
// unused indices 14 and 15.
constexpr int triple_digit(int idx, int d) {
    if (idx > 13) return 0;
    const int d2 = (idx + 1) % 3 - 1;
    const int rest = (idx - d2) / 3;
    const int d1 = (rest + 1) % 3 - 1;
    const int d0 = (rest - d1) / 3;
    return d == 0 ? d0 : d == 1 ? d1 : d2;
}

constexpr uint32_t byte_of(int v, int pos) { return ((uint32_t)v & 0xFFu) << (8 * pos); }

// The two expansion tables as one constant image (computed at compile time), copied into LDS by each work group:
// index-table entry e (two words) for index byte e & 255 and sign bits e >> 8, then the 256 pair-table words.
struct ExpandTables {
    uint32_t w[kTl2MfmaTables / 4];
    constexpr ExpandTables() : w{} {
        for (int e = 0; e < 1024; ++e) {
            const int n0 = e & 15, n1 = (e >> 4) & 15;
            const int g0 = (e >> 8) & 1 ? -1 : 1, g1 = (e >> 9) & 1 ? -1 : 1;
            w[2 * e] = byte_of(g0 * triple_digit(n0, 0), 0) | byte_of(g0 * triple_digit(n0, 1), 1) |
                       byte_of(g0 * triple_digit(n0, 2), 2) | byte_of(g1 * triple_digit(n1, 0), 3);
            w[2 * e + 1] = byte_of(g1 * triple_digit(n1, 1), 0) | byte_of(g1 * triple_digit(n1, 2), 1);
        }
        for (int b = 0; b < 256; ++b) {
            const int c0 = b & 15, c1 = b >> 4;
            uint32_t v = 0;
            if (c0 <= 8) v |= byte_of(c0 / 3 - 1, 0) | byte_of(c0 % 3 - 1, 1);
            if (c1 <= 8) v |= byte_of(c1 / 3 - 1, 2) | byte_of(c1 % 3 - 1, 3);
            w[2048 + b] = v;
        }
    }
};
__device__ __align__(16) constexpr ExpandTables kExpandTables{};
constexpr int kTableChunks = kTl2MfmaTables / 16;              // 16-byte chunks of the image

// The 96 weights of a lane's 32 triples (index words iw, sign word sw) as 24 words, k in order.
__device__ __forceinline__ void expand_triples(const v4u& iw, uint32_t sw, const uint2* itab, uint32_t (&wd)[24]) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t w = word_of(iw, j);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int p = 4 * j + 2 * h;                 // bytes p, p + 1: triples 2p .. 2p + 3
            const uint32_t i0 = ((w >> (16 * h)) & 0xFFu) | (((sw >> (2 * p)) & 3u) << 8);
            const uint32_t i1 = ((w >> (16 * h + 8)) & 0xFFu) | (((sw >> (2 * p + 2)) & 3u) << 8);
            const uint2 e0 = itab[i0], e1 = itab[i1];
            const int d = 6 * j + 3 * h;
            wd[d] = e0.x;
            wd[d + 1] = e0.y | (e1.x << 16);
            wd[d + 2] = (e1.x >> 16) | (e1.y << 16);
        }
    }
}

// XV = 0: the codes and scales are read (xq, x_scale).  XV > 0: one token (M = 1), its fp32 row x quantised here
// (Sec. 2.1; XV float4 per thread), as in the single-token I2_S kernel: the row is loaded before the first weights,
// reduced to its absmax through LDS and converted into the LDS codes; work group 0 writes xq, x_scale, x_rowsum.
//
// MB (K past 48 blocks): a row group takes nb = ceil(nblk / (WAVES U)) batches of WAVES U blocks, walked as the steps
// of the stream (the accumulators carry over a row group's batches; its last batch holds the TL1 tail and the
// reduction), and the codes of every token are copied whole into LDS.
template <int WAVES, int U, int CH, int XV, bool MB>
__global__ __launch_bounds__(64 * WAVES) void tl2_mfma_decode_kernel(FusedLinears L, const float* __restrict__ x,
                                                                     int8_t* xq, float* x_scale,
                                                                     int32_t* x_rowsum, int M, int K) {
    extern __shared__ __align__(16) uint8_t lds[];    // index table | pair table | M rows of K + 16 codes
    __shared__ v4i part[2][WAVES][64];
    __shared__ float redf[WAVES];
    __shared__ int redi[WAVES];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q = lane >> 4, r = lane & 15;
    const int G = gridDim.x, bid = blockIdx.x;
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    const int nblk = three / kTl2BlockK;                       // >= 1 (the launcher checks)
    const int units = (K - three) / kSubK;
    const int tail_wave = nblk % WAVES;                        // a wave with the fewest blocks
    constexpr int kPerBatch = WAVES * U;
    const int nb = MB ? (nblk + kPerBatch - 1) / kPerBatch : 1;  // batches per row group
    const int S = ((L.total - bid + G - 1) / G) * nb;          // steps of this work group (grid <= total)
    // step st = batch b of row group g
    auto step_gb = [&](int st, int& g, int& b) {
        const int gi = MB ? st / nb : st;
        b = MB ? st - gi * nb : 0;
        g = bid + gi * G;
    };
    const int stride = K + 16;
    const uint2* itab = reinterpret_cast<const uint2*>(lds);
    const uint32_t* ptab = reinterpret_cast<const uint32_t*>(lds + kIdxTableBytes);
    int8_t* xs = reinterpret_cast<int8_t*>(lds + kTl2MfmaTables);

    // the loads of row group step st, all unconditional (blocks past nblk repeat a real one; the tail words of
    // waves other than the tail wave, and of units past `units`, repeat one real word)
    const bool tail_mine = wave == tail_wave && units > 0;
    auto issue = [&](v4u (&iw)[U], uint32_t (&sw)[U], uint32_t (&tw)[kMaxUnits], float& bw, int st) {
        int g, b, li, rg;
        step_gb(st, g, b);
        locate(L, g, li, rg);
        const size_t Nl = (size_t)pick(L.N, li);
        const uint8_t* idx_plane = pick(L.packed, li);
        const uint8_t* sign_plane = idx_plane + Nl * (three / 6);
        const uint8_t* tail_plane = sign_plane + Nl * (three / 24);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t tile = (size_t)rg * nblk + min(b * kPerBatch + wave + WAVES * u, nblk - 1);
            iw[u] = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(idx_plane + tile * 1024 + 16 * lane));
            sw[u] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(sign_plane + tile * 256 + 4 * lane));
        }
        const int um = units > 0 ? units : 1;
        const uint8_t* tail_base = units > 0 ? tail_plane : idx_plane;
        const size_t tail_row = tail_mine ? (size_t)rg * 64 * um + (size_t)lane * um : 0;
#pragma unroll
        for (int t = 0; t < kMaxUnits; ++t)
            tw[t] = *reinterpret_cast<const uint32_t*>(tail_base + (tail_row + (tail_mine ? min(t, um - 1) : 0)) * 4);
        bw = *pick(L.w_scale, li);
    };

    // epilogue operands of tokens m = 4q + v (XV > 0: the scale computed below)
    float xs_m[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) xs_m[v] = (XV == 0 && 4 * q + v < M) ? x_scale[4 * q + v] : 1.0f;

    // the expansion tables: chunk tid + 64 WAVES i of the constant image, loaded first, stored into LDS later
    constexpr int kTabPer = (kTableChunks + 64 * WAVES - 1) / (64 * WAVES);
    v4u tabv[kTabPer];
    auto load_tables = [&]() {
#pragma unroll
        for (int i = 0; i < kTabPer; ++i)
            tabv[i] = reinterpret_cast<const v4u*>(kExpandTables.w)[min(tid + 64 * WAVES * i, kTableChunks - 1)];
    };
    auto store_tables = [&]() {
#pragma unroll
        for (int i = 0; i < kTabPer; ++i)
            if (tid + 64 * WAVES * i < kTableChunks) reinterpret_cast<v4u*>(lds)[tid + 64 * WAVES * i] = tabv[i];
    };

    // this wave's codes: 24 chunks of 16 bytes per token and block (4 per token and tail unit); CH chunks per lane
    // and block cover 64 CH / 24 tokens.  Loads issued before the first weights are usable before those arrive
    // (loads complete in order); the stores follow the tables.
    constexpr int kChunks = CH;
    v4i cc[XV == 0 ? U : 1][kChunks];
    auto load_codes = [&]() {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int blk = min(wave + WAVES * u, nblk - 1);
#pragma unroll
            for (int i = 0; i < kChunks; ++i) {
                const int ch = min(lane + 64 * i, M * 24 - 1);
                const int m = ch / 24, k = blk * kTl2BlockK + 16 * (ch % 24);
                cc[u][i] = *reinterpret_cast<const v4i*>(xq + (size_t)m * K + k);
            }
        }
    };
    auto store_codes = [&]() {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int blk = wave + WAVES * u;
#pragma unroll
            for (int i = 0; i < kChunks; ++i) {
                const int ch = lane + 64 * i;
                if (blk < nblk && ch < M * 24) {
                    const int m = ch / 24, k = blk * kTl2BlockK + 16 * (ch % 24);
                    *reinterpret_cast<v4i*>(xs + m * stride + k) = cc[u][i];
                }
            }
        }
        if (tail_mine) {
            for (int ch = lane; ch < M * 4 * units; ch += 64) {
                const int m = ch / (4 * units), k = three + 16 * (ch % (4 * units));
                *reinterpret_cast<v4i*>(xs + m * stride + k) = *reinterpret_cast<const v4i*>(xq + (size_t)m * K + k);
            }
        }
    };
    // one token: the fp32 row, float4 e = tid + 64 WAVES i per thread
    constexpr int kXv = XV > 0 ? XV : 1;
    float4 xv[kXv];
    const int K4 = K >> 2;
    auto load_row = [&]() {
#pragma unroll
        for (int i = 0; i < kXv; ++i) {
            const int e = tid + i * 64 * WAVES;
            const float4 v = reinterpret_cast<const float4*>(x)[e < K4 ? e : K4 - 1];
            xv[i] = e < K4 ? v : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
    };
    auto quantise_row = [&]() {
        float amax = 0.0f;
#pragma unroll
        for (int i = 0; i < kXv; ++i)
            amax = fmaxf(amax, fmaxf(fmaxf(fabsf(xv[i].x), fabsf(xv[i].y)), fmaxf(fabsf(xv[i].z), fabsf(xv[i].w))));
        amax = wave_max_all(amax);
        if (lane == 0) redf[wave] = amax;
        __syncthreads();
        amax = redf[0];
#pragma unroll
        for (int w = 1; w < WAVES; ++w) amax = fmaxf(amax, redf[w]);
        const float sx = 127.0f / fmaxf(amax, 1e-5f);
        int sum = 0;
#pragma unroll
        for (int i = 0; i < kXv; ++i) {
            const int e = tid + i * 64 * WAVES;
            if (e < K4) {
                const uint32_t c = quant4(xv[i], sx);
                sum = byte_sum4(c, sum);
                reinterpret_cast<uint32_t*>(xs)[e] = c;
                if (bid == 0) reinterpret_cast<uint32_t*>(xq)[e] = c;
            }
        }
        sum = wave_sum_all(sum);
        if (lane == 0) redi[wave] = sum;
        xs_m[0] = sx;
        if (bid == 0 && tid == 0) x_scale[0] = sx;
    };

    const v4i zero = {0, 0, 0, 0};
    const int8_t* arow = xs + (r < M ? r : 0) * stride;
    int par = 0;
    v4i acc = zero;
    auto compute = [&](const v4u (&iw)[U], const uint32_t (&sw)[U], const uint32_t (&tw)[kMaxUnits], float bw,
                       int st) {
        int g, b;
        step_gb(st, g, b);
        if (b == 0) acc = zero;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int blk = b * kPerBatch + wave + WAVES * u;
            if (blk < nblk) {
                uint32_t wd[24];
                expand_triples(iw[u], sw[u], itab, wd);
                const int8_t* ab = arow + blk * kTl2BlockK + 96 * q;
#pragma unroll
                for (int s6 = 0; s6 < 6; ++s6) {
                    const v4i b = {(int)wd[4 * s6], (int)wd[4 * s6 + 1], (int)wd[4 * s6 + 2], (int)wd[4 * s6 + 3]};
                    acc = mfma16x16x64(*reinterpret_cast<const v4i*>(ab + 16 * s6), b, acc);
                }
            }
        }
        if (b < nb - 1) return;      // the row group's last batch: the tail and the reduction
        if (tail_mine) {
#pragma unroll
            for (int t = 0; t < kMaxUnits; ++t) {
                if (t < units) {
                    const uint32_t w = tw[t];
                    const v4i b = {(int)ptab[w & 0xFFu], (int)ptab[(w >> 8) & 0xFFu], (int)ptab[(w >> 16) & 0xFFu],
                                   (int)ptab[w >> 24]};
                    acc = mfma16x16x64(*reinterpret_cast<const v4i*>(arow + three + kSubK * t + 16 * q), b, acc);
                }
            }
        }
        part[par][wave][lane] = acc;
        __syncthreads();
        if (wave == 0 && 4 * q < M) {
            v4i tot = part[par][0][lane];
#pragma unroll 4
            for (int w2 = 1; w2 < WAVES; ++w2) tot += part[par][w2][lane];
            int li, rg;
            locate(L, g, li, rg);
            const int N = pick(L.N, li);
            const int n = rg * kRowsPerGroup + r;
            float* y = pick(L.y, li);
            int32_t* acc_out = pick(L.acc, li);
            // D element v of lane l is row 4 (l / 16) + v (token), column l % 16 (weight row)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = 4 * q + v;
                if (m < M) {
                    y[(size_t)m * N + n] = (float)tot[v] * (bw / xs_m[v]);
                    if (acc_out) acc_out[(size_t)m * N + n] = tot[v];
                }
            }
        }
        par ^= 1;
    };

    // one and several row groups per work group are separate instantiations, so no two paths with different
    // loads in flight join
    auto run = [&](auto multi) {
        constexpr bool kMulti = decltype(multi)::value;
        v4u iwa[U], iwb[U];
        uint32_t swa[U], swb[U], twa[kMaxUnits], twb[kMaxUnits];
        float ba = 0.0f, bb = 0.0f;
        // codes loaded ahead of the weights where their registers fit beside them (one token-group of chunks per
        // wave), after them otherwise
        constexpr bool kEarly = XV == 0 && !MB && U * CH <= 3;
        load_tables();
        if constexpr (XV > 0) load_row();
        else if constexpr (kEarly) load_codes();
        // every wave's row (or code) loads enter the memory pipeline before any weight load, so that no wave's
        // activation waits behind the other waves' weight batches
        if constexpr (XV > 0 || kEarly) __builtin_amdgcn_s_barrier();
        // two batches in flight from the start when the codes are given; one while the row is quantised (a second
        // batch ahead of the quantisation delays the row's arrival more than it saves later), the second after it
        issue(iwa, swa, twa, ba, 0);
        if constexpr (kMulti && XV == 0) issue(iwb, swb, twb, bb, 1);
        __builtin_amdgcn_sched_barrier(0);   // keep the weight loads ahead of the tables and the conversion
        if constexpr (XV == 0 && !MB && !kEarly) load_codes();
        store_tables();
        if constexpr (XV > 0) {
            quantise_row();
            if constexpr (kMulti) issue(iwb, swb, twb, bb, 1);
        } else if constexpr (MB) {
            // every token's codes, whole (16-byte chunks; K % 64 == 0)
            const int kc = K / 16;
            for (int ch = tid; ch < M * kc; ch += 64 * WAVES) {
                const int m = ch / kc, k = 16 * (ch - m * kc);
                *reinterpret_cast<v4i*>(xs + m * stride + k) = *reinterpret_cast<const v4i*>(xq + (size_t)m * K + k);
            }
        } else {
            store_codes();
        }
        __syncthreads();                                   // the tables (and codes) are shared by every wave
        if (XV > 0 && bid == 0 && tid == 0) {
            int tot = 0;
            for (int w = 0; w < WAVES; ++w) tot += redi[w];
            x_rowsum[0] = tot;
        }
        if constexpr (!kMulti) {
            compute(iwa, swa, twa, ba, 0);
            return;
        }
        int st = 0;
        for (; st + 3 < S; st += 2) {
            compute(iwa, swa, twa, ba, st);
            issue(iwa, swa, twa, ba, st + 2);
            compute(iwb, swb, twb, bb, st + 1);
            issue(iwb, swb, twb, bb, st + 3);
        }
        if (st + 2 < S) {
            compute(iwa, swa, twa, ba, st);
            issue(iwa, swa, twa, ba, st + 2);
            compute(iwb, swb, twb, bb, st + 1);
            compute(iwa, swa, twa, ba, st + 2);
        } else {
            compute(iwa, swa, twa, ba, st);
            compute(iwb, swb, twb, bb, st + 1);
        }
    };
    if (S == 1) run(std::false_type{});
    else run(std::true_type{});
}

// The weights of one transcoding launch.  Pair items (two TL2 blocks of one row group) of weight i are numbered
// from pstart[i], its work groups of single items from rstart[i] (LLONG_MAX past the last weight).
struct TranscodeLinears {
    const uint8_t* packed[kMaxFused];
    uint32_t* out[kMaxFused];
    int N[kMaxFused];
    long long pstart[kMaxFused];
    long long rstart[kMaxFused];
    long long pairs;                  // pair items of the launch
    int pair_groups;                  // persistent work groups that walk them
};

// TL2 -> I2_S transcoding, for the prefill GEMM (M > 16): the I2_S MFMA GEMM then runs on the same ternary
// weights.  A lane expands its 32 triples (one row, 96 consecutive k of a 384-k block) through the expansion
// tables as the MFMA decode kernel does and writes them as six I2_S words: the word of row n and k0 (a multiple
// of 16) holds code t + 1 of k = k0 + 4f + b in bits 2f + 8b, at word R K + 256 s + l T + j of the I2_S array
// (R = n / 16, block s = k0 / 256, sub-tile j = (k0 mod 256) / 64, lane chunk l = 16 ((k0 mod 64) / 16) + n mod 16,
// T = the block's sub-tiles).  Tail units (TL1 pairs, Table 5) give one word per lane each.
__device__ __forceinline__ uint32_t i2s_word_of(const uint32_t* d) {
    // t in {-1, 0, 1} per byte -> code t + 1 in the low two bits of each byte
    uint32_t w = 0;
#pragma unroll
    for (int f = 0; f < 4; ++f) w |= (((d[f] & 0x03030303u) + 0x01010101u) & 0x03030303u) << (2 * f);
    return w;
}

__device__ __forceinline__ size_t i2s_word_index(int n, int k0, int K) {
    const int R = n / kRowsPerGroup, r = n % kRowsPerGroup;
    const int sb = k0 / kI2sBlockK, rem = k0 % kI2sBlockK;
    const int j = rem / kSubK, q = (rem % kSubK) / 16;
    const int T = min(4, K / kSubK - 4 * sb);
    return (size_t)R * K + (size_t)kI2sBlockK * sb + (size_t)(16 * q + r) * T + j;
}

// Work groups of 192 threads.  The first T.pair_groups groups walk the pair items p = blockIdx.x, + gridDim, ...: a
// pair is two TL2 blocks of one row group, 768 k, exactly three full I2_S blocks (one contiguous 3 KiB run of the
// I2_S array).  Two waves expand its 128 lane chunks into LDS at the words' places in that run, then the three
// waves store the run with one 16-byte store per thread, while the next pair's packed words are already in
// flight.  The other groups take one item per thread: the lane chunks of an odd last TL2 block and the tail
// words, written word by word.  The packed words are loaded before the table image is copied into LDS.
constexpr int kTcThreads = 192;

__device__ __forceinline__ void tc_counts(int N, int K, long long& pairs, long long& odd_items,
                                          long long& rest_items) {
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    const int nblk = three / kTl2BlockK, units = (K - three) / kSubK;
    const long long rgs = N / kRowsPerGroup;
    pairs = rgs * (nblk / 2);
    odd_items = rgs * 64 * (nblk & 1);
    rest_items = odd_items + rgs * 64 * units;
}

__global__ __launch_bounds__(kTcThreads) void tl2_to_i2s_kernel(TranscodeLinears T, int K) {
    __shared__ __align__(16) uint8_t tab[kTl2MfmaTables];
    __shared__ __align__(16) uint32_t run[3 * kI2sBlockK];     // one pair's three I2_S blocks, as in HBM
    const int tid = threadIdx.x;
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    const int nblk = three / kTl2BlockK;
    const int units = (K - three) / kSubK;
    const int l = tid & 63, q = l >> 4, r = l & 15;
    auto planes = [&](int li, const uint8_t*& idx_plane, const uint8_t*& sign_plane, const uint8_t*& tail_plane) {
        const size_t N = (size_t)T.N[li];
        idx_plane = T.packed[li];
        sign_plane = idx_plane + N * (three / 6);
        tail_plane = sign_plane + N * (three / 24);
    };
    auto copy_tables = [&]() {
        for (int i = tid; i < kTableChunks; i += kTcThreads)
            reinterpret_cast<v4u*>(tab)[i] = reinterpret_cast<const v4u*>(kExpandTables.w)[i];
    };

    if ((int)blockIdx.x < T.pair_groups) {
        const int pairs_rg = nblk / 2;
        // pair p: weight li, row group R, pair pp within the row group
        auto locate_pair = [&](long long p, int& li, int& R, int& pp) {
            li = 0;
#pragma unroll
            for (int i = 1; i < kMaxFused; ++i) li = p >= T.pstart[i] ? i : li;
            const long long b = p - T.pstart[li];
            R = (int)(b / pairs_rg);
            pp = (int)(b - (long long)R * pairs_rg);
        };
        // this lane's packed words of pair p (waves 0 and 1: blocks 2 pp and 2 pp + 1; wave 2 loads nothing)
        auto load_pair = [&](long long p, v4u& iw, uint32_t& sw) {
            int li, R, pp;
            locate_pair(p, li, R, pp);
            const uint8_t *ip, *sp, *tp;
            planes(li, ip, sp, tp);
            const size_t tile = (size_t)R * nblk + 2 * pp + (tid >> 6);
            iw = *reinterpret_cast<const v4u*>(ip + tile * 1024 + 16 * l);
            sw = *reinterpret_cast<const uint32_t*>(sp + tile * 256 + 4 * l);
        };
        long long p = blockIdx.x;
        const long long G = T.pair_groups;
        v4u iw = {0u, 0u, 0u, 0u};
        uint32_t sw = 0u;
        if (tid < 128 && p < T.pairs) load_pair(p, iw, sw);
        copy_tables();
        __syncthreads();
        for (; p < T.pairs; p += G) {
            v4u iw_n = {0u, 0u, 0u, 0u};
            uint32_t sw_n = 0u;
            if (tid < 128 && p + G < T.pairs) load_pair(p + G, iw_n, sw_n);
            int li, R, pp;
            locate_pair(p, li, R, pp);
            if (tid < 128) {
                uint32_t wd[24];
                expand_triples(iw, sw, reinterpret_cast<const uint2*>(tab), wd);
                // word (block s, lane chunk 16 qq + r, sub-tile j) of the run, relative to its first k (768 pp)
                const int base = (tid >> 6) * kTl2BlockK + 96 * q;
#pragma unroll
                for (int g = 0; g < 6; ++g) {
                    const int kk = base + 16 * g;
                    const int s_l = kk / kI2sBlockK, rem = kk % kI2sBlockK;
                    run[kI2sBlockK * s_l + (16 * ((rem % kSubK) / 16) + r) * 4 + rem / kSubK] = i2s_word_of(wd + 4 * g);
                }
            }
            __syncthreads();
            const size_t first = (size_t)R * K + (size_t)pp * 2 * kTl2BlockK;   // words: 768 pp of row group R
            reinterpret_cast<v4u*>(T.out[li] + first)[tid] = reinterpret_cast<const v4u*>(run)[tid];
            __syncthreads();                                   // the run is rewritten by the next pair
            iw = iw_n;
            sw = sw_n;
        }
        return;
    }

    // single items: group rb of weight li
    const long long rb_all = (long long)blockIdx.x - T.pair_groups;
    int li = 0;
#pragma unroll
    for (int i = 1; i < kMaxFused; ++i) li = rb_all >= T.rstart[i] ? i : li;
    long long pairs, odd_items, rest_items;
    tc_counts(T.N[li], K, pairs, odd_items, rest_items);
    const uint8_t *idx_plane, *sign_plane, *tail_plane;
    planes(li, idx_plane, sign_plane, tail_plane);
    uint32_t* __restrict__ out = T.out[li];
    const long long c = (rb_all - T.rstart[li]) * kTcThreads + tid;
    int R = 0, lc = 0, u = 0;
    bool expand = false, tail = false;
    if (c < odd_items) {
        R = (int)(c >> 6);
        lc = (int)(c & 63);
        expand = true;
    } else if (c < rest_items) {
        const long long t = c - odd_items;                     // (row group, lane, unit), as the tail plane
        u = (int)(t % units);
        lc = (int)((t / units) & 63);
        R = (int)(t / ((long long)64 * units));
        tail = true;
    }
    v4u iw = {0u, 0u, 0u, 0u};
    uint32_t sw = 0u, tw = 0u;
    if (expand) {
        const size_t tile = (size_t)R * nblk + nblk - 1;
        iw = *reinterpret_cast<const v4u*>(idx_plane + tile * 1024 + 16 * lc);
        sw = *reinterpret_cast<const uint32_t*>(sign_plane + tile * 256 + 4 * lc);
    } else if (tail) {
        tw = *reinterpret_cast<const uint32_t*>(tail_plane + ((size_t)R * 64 * units + (size_t)lc * units + u) * 4);
    }
    copy_tables();
    __syncthreads();
    const int qc = lc >> 4, n = R * kRowsPerGroup + (lc & 15);
    if (expand) {
        uint32_t wd[24];
        expand_triples(iw, sw, reinterpret_cast<const uint2*>(tab), wd);
        const int base = (nblk - 1) * kTl2BlockK + 96 * qc;
#pragma unroll
        for (int g = 0; g < 6; ++g) out[i2s_word_index(n, base + 16 * g, K)] = i2s_word_of(wd + 4 * g);
    } else if (tail) {
        const uint32_t* ptab = reinterpret_cast<const uint32_t*>(tab + kIdxTableBytes);
        const uint32_t d[4] = {ptab[tw & 0xFFu], ptab[(tw >> 8) & 0xFFu], ptab[(tw >> 16) & 0xFFu], ptab[tw >> 24]};
        out[i2s_word_index(n, three + kSubK * u + 16 * qc, K)] = i2s_word_of(d);
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
    // Each wave holds the tables of a chunk of tokens (kTokenStride bytes each); stay within the LDS budget.
    const int tc = tl2_elut_chunk(M);
    int w = 16;
    while (w > 1 && (size_t)w * tc * kTokenStride > (size_t)kElutLdsBudget) w >>= 1;
    return w;
}

size_t tl2_elut_lds_bytes(int M) {
    const size_t tables = (size_t)tl2_elut_waves(M) * tl2_elut_chunk(M) * kTokenStride;
    const size_t red = (size_t)tl2_elut_waves(M) * 16 * 16 * sizeof(int);
    return tables > red ? tables : red;
}

// Arguments of one table-lookup launch over a fused weight group; x set: one token quantised inside (QX).
struct LookupArgs {
    const FusedLinears* L;
    const float* x;
    const int8_t* xq;
    const float* x_scale;
    int M, K;
    int8_t* xq_out;
    float* s_out;
    int32_t* rs_out;
};

template <int WAVES, int MT, bool LOSSY, bool QX>
void launch_tl2_cfg(const LookupArgs& a, size_t lds, hipStream_t stream) {
    hipLaunchKernelGGL((tl2_elut_decode_kernel<WAVES, MT, LOSSY, QX>), dim3((unsigned)a.L->total), dim3(64 * WAVES),
                       lds, stream, *a.L, a.x, a.xq, a.x_scale, a.M, a.K, a.xq_out, a.s_out, a.rs_out);
}

template <int MT, bool LOSSY, bool QX>
hipError_t launch_elut_mt(const LookupArgs& a, hipStream_t stream) {
    const size_t lds = tl2_elut_lds_bytes(a.M);
    switch (tl2_elut_waves(a.M)) {
        case 16: launch_tl2_cfg<16, MT, LOSSY, QX>(a, lds, stream); break;
        case 8: launch_tl2_cfg<8, MT, LOSSY, QX>(a, lds, stream); break;
        case 4: launch_tl2_cfg<4, MT, LOSSY, QX>(a, lds, stream); break;
        case 2: launch_tl2_cfg<2, MT, LOSSY, QX>(a, lds, stream); break;
        default: launch_tl2_cfg<1, MT, LOSSY, QX>(a, lds, stream); break;
    }
    return hipGetLastError();
}

template <bool LOSSY>
hipError_t launch_tl2_elut_lossy(const LookupArgs& a, hipStream_t stream) {
    if (a.x) return launch_elut_mt<1, LOSSY, true>(a, stream);
    if (a.M <= 1) return launch_elut_mt<1, LOSSY, false>(a, stream);
    if (a.M <= 2) return launch_elut_mt<2, LOSSY, false>(a, stream);
    if (a.M <= 4) return launch_elut_mt<4, LOSSY, false>(a, stream);
    return launch_elut_mt<8, LOSSY, false>(a, stream);
}

hipError_t launch_tl2_elut_decode(const FusedLinears& L, const float* x, const int8_t* xq, const float* x_scale,
                                  int M, int K, int8_t* xq_out, float* s_out, int32_t* rs_out, hipStream_t stream,
                                  bool lossy) {
    if (L.total <= 0) return hipSuccess;
    if (M < 1 || M > 8 || (x && M != 1)) return hipErrorInvalidValue;
    const LookupArgs a{&L, x, xq, x_scale, M, K, xq_out, s_out, rs_out};
    return lossy ? launch_tl2_elut_lossy<true>(a, stream) : launch_tl2_elut_lossy<false>(a, stream);
}

// TL1 layout by table lookup (Algorithm TL1): the 32 pair tables of a 64-k unit per wave, lossy or not.
int tl1_elut_waves(int M) {
    const int tc = tl2_elut_chunk(M);
    int w = 16;
    while (w > 1 && (size_t)w * tc * kTl1BlockStride > (size_t)kElutLdsBudget) w >>= 1;
    return w;
}

size_t tl1_elut_lds_bytes(int M) {
    const size_t tables = (size_t)tl1_elut_waves(M) * tl2_elut_chunk(M) * kTl1BlockStride;
    const size_t red = (size_t)tl1_elut_waves(M) * 16 * 16 * sizeof(int);
    return tables > red ? tables : red;
}

template <int WAVES, int MT, bool LOSSY, bool QX>
void launch_tl1_cfg(const LookupArgs& a, size_t lds, hipStream_t stream) {
    hipLaunchKernelGGL((tl1_elut_decode_kernel<WAVES, MT, LOSSY, QX>), dim3((unsigned)a.L->total), dim3(64 * WAVES),
                       lds, stream, *a.L, a.x, a.xq, a.x_scale, a.M, a.K, a.xq_out, a.s_out, a.rs_out);
}

template <int MT, bool LOSSY, bool QX>
hipError_t launch_tl1_mt(const LookupArgs& a, hipStream_t stream) {
    const size_t lds = tl1_elut_lds_bytes(a.M);
    switch (tl1_elut_waves(a.M)) {
        case 16: launch_tl1_cfg<16, MT, LOSSY, QX>(a, lds, stream); break;
        case 8: launch_tl1_cfg<8, MT, LOSSY, QX>(a, lds, stream); break;
        default: launch_tl1_cfg<4, MT, LOSSY, QX>(a, lds, stream); break;
    }
    return hipGetLastError();
}

template <bool LOSSY>
hipError_t launch_tl1_elut_lossy(const LookupArgs& a, hipStream_t stream) {
    if (a.x) return launch_tl1_mt<1, LOSSY, true>(a, stream);
    if (a.M <= 1) return launch_tl1_mt<1, LOSSY, false>(a, stream);
    if (a.M <= 2) return launch_tl1_mt<2, LOSSY, false>(a, stream);
    if (a.M <= 4) return launch_tl1_mt<4, LOSSY, false>(a, stream);
    return launch_tl1_mt<8, LOSSY, false>(a, stream);
}

hipError_t launch_tl1_elut_decode(const FusedLinears& L, const float* x, const int8_t* xq, const float* x_scale,
                                  int M, int K, int8_t* xq_out, float* s_out, int32_t* rs_out, hipStream_t stream,
                                  bool lossy) {
    if (L.total <= 0) return hipSuccess;
    if (M < 1 || M > 8 || (x && M != 1)) return hipErrorInvalidValue;
    const LookupArgs a{&L, x, xq, x_scale, M, K, xq_out, s_out, rs_out};
    return lossy ? launch_tl1_elut_lossy<true>(a, stream) : launch_tl1_elut_lossy<false>(a, stream);
}

size_t tl2_stream_lds_bytes(int K) {
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    return (size_t)((K + 15) & ~15) + (size_t)(three / kTl2BlockK) * kBlockBytes28 +
           (size_t)((K - three) / kSubK) * 32 * kSlot28;
}

bool tl2_stream_fits(int K) {
    return K >= kTl2BlockK && tl2_stream_lds_bytes(K) + 2 * 16 * 16 * 4 + 256 <= 160 * 1024;
}

template <int WAVES, int U, int XV, bool LOSSY>
hipError_t launch_stream_cfg(const FusedLinears& L, const float* x, int K, int8_t* xq, float* s, int32_t* rs,
                             hipStream_t stream) {
    const size_t lds = tl2_stream_lds_bytes(K);
    const void* kern = x ? reinterpret_cast<const void*>(tl2_stream_kernel<WAVES, U, XV, true, LOSSY>)
                         : reinterpret_cast<const void*>(tl2_stream_kernel<WAVES, U, XV, false, LOSSY>);
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, 64 * WAVES, lds) != hipSuccess || occ <= 0) occ = 1;
    const int64_t max_g = (int64_t)device_cus() * occ;
    const int64_t rounds = (L.total + max_g - 1) / max_g;
    const dim3 grid((unsigned)((L.total + rounds - 1) / rounds)), block(64 * WAVES);
    if (x)
        hipLaunchKernelGGL((tl2_stream_kernel<WAVES, U, XV, true, LOSSY>), grid, block, lds, stream, L, x, K, xq, s,
                           rs);
    else
        hipLaunchKernelGGL((tl2_stream_kernel<WAVES, U, XV, false, LOSSY>), grid, block, lds, stream, L, x, K, xq, s,
                           rs);
    return hipGetLastError();
}

template <int WAVES, int U, bool LOSSY>
hipError_t launch_stream_u(const FusedLinears& L, const float* x, int K, int8_t* xq, float* s, int32_t* rs,
                           hipStream_t stream) {
    const int xv = (K / 4 + 64 * WAVES - 1) / (64 * WAVES);
    if (xv <= 1) return launch_stream_cfg<WAVES, U, 1, LOSSY>(L, x, K, xq, s, rs, stream);
    if (xv <= 2) return launch_stream_cfg<WAVES, U, 2, LOSSY>(L, x, K, xq, s, rs, stream);
    if (xv <= 4) return launch_stream_cfg<WAVES, U, 4, LOSSY>(L, x, K, xq, s, rs, stream);
    return launch_stream_cfg<WAVES, U, 8, LOSSY>(L, x, K, xq, s, rs, stream);
}

template <bool LOSSY>
hipError_t launch_tl2_stream_t(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                               int32_t* x_rowsum, hipStream_t stream) {
    const int nblk = K / kTl2BlockK;
    if (nblk <= 4) return launch_stream_u<4, 1, LOSSY>(L, x, K, xq, x_scale, x_rowsum, stream);
    if (nblk <= 8) return launch_stream_u<8, 1, LOSSY>(L, x, K, xq, x_scale, x_rowsum, stream);
    if (nblk <= 16) return launch_stream_u<8, 2, LOSSY>(L, x, K, xq, x_scale, x_rowsum, stream);
    if (nblk <= 32) return launch_stream_u<16, 2, LOSSY>(L, x, K, xq, x_scale, x_rowsum, stream);
    return launch_stream_u<16, 3, LOSSY>(L, x, K, xq, x_scale, x_rowsum, stream);
}

// Waves and blocks per wave: every block of a row has its wave (at most three per wave).
hipError_t launch_tl2_stream(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                             int32_t* x_rowsum, hipStream_t stream, bool lossy) {
    return lossy ? launch_tl2_stream_t<true>(L, x, K, xq, x_scale, x_rowsum, stream)
                 : launch_tl2_stream_t<false>(L, x, K, xq, x_scale, x_rowsum, stream);
}

size_t tl1_stream_lds_bytes(int K) {
    return (size_t)((K + 15) & ~15) + (size_t)((K / kSubK + 3) / 4) * kTl1BlockBytes20;
}

bool tl1_stream_fits(int K) {
    const int nkb = (K / kSubK + 3) / 4;
    return K >= kSubK && nkb <= 64 && tl1_stream_lds_bytes(K) + 2 * 16 * 16 * 4 + 256 <= 160 * 1024;
}

template <int WAVES, int U, int XV>
hipError_t launch_tl1_stream_cfg(const FusedLinears& L, const float* x, int K, int8_t* xq, float* s, int32_t* rs,
                                 hipStream_t stream) {
    const size_t lds = tl1_stream_lds_bytes(K);
    const void* kern = x ? reinterpret_cast<const void*>(tl1_lossy_stream_kernel<WAVES, U, XV, true>)
                         : reinterpret_cast<const void*>(tl1_lossy_stream_kernel<WAVES, U, XV, false>);
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, 64 * WAVES, lds) != hipSuccess || occ <= 0) occ = 1;
    const int64_t max_g = (int64_t)device_cus() * occ;
    const int64_t rounds = (L.total + max_g - 1) / max_g;
    const dim3 grid((unsigned)((L.total + rounds - 1) / rounds)), block(64 * WAVES);
    if (x)
        hipLaunchKernelGGL((tl1_lossy_stream_kernel<WAVES, U, XV, true>), grid, block, lds, stream, L, x, K, xq, s, rs);
    else
        hipLaunchKernelGGL((tl1_lossy_stream_kernel<WAVES, U, XV, false>), grid, block, lds, stream, L, x, K, xq, s,
                           rs);
    return hipGetLastError();
}

template <int WAVES, int U>
hipError_t launch_tl1_stream_u(const FusedLinears& L, const float* x, int K, int8_t* xq, float* s, int32_t* rs,
                               hipStream_t stream) {
    const int xv = (K / 4 + 64 * WAVES - 1) / (64 * WAVES);
    if (xv <= 1) return launch_tl1_stream_cfg<WAVES, U, 1>(L, x, K, xq, s, rs, stream);
    if (xv <= 2) return launch_tl1_stream_cfg<WAVES, U, 2>(L, x, K, xq, s, rs, stream);
    if (xv <= 4) return launch_tl1_stream_cfg<WAVES, U, 4>(L, x, K, xq, s, rs, stream);
    return launch_tl1_stream_cfg<WAVES, U, 8>(L, x, K, xq, s, rs, stream);
}

// Waves and blocks per wave: every 256-k block of the row has its wave (at most four per wave).
hipError_t launch_tl1_lossy_stream(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                                   int32_t* x_rowsum, hipStream_t stream) {
    if (!tl1_stream_fits(K)) return hipErrorInvalidValue;
    const int nkb = (K / kSubK + 3) / 4;
    if (nkb <= 4) return launch_tl1_stream_u<4, 1>(L, x, K, xq, x_scale, x_rowsum, stream);
    if (nkb <= 8) return launch_tl1_stream_u<8, 1>(L, x, K, xq, x_scale, x_rowsum, stream);
    if (nkb <= 16) return launch_tl1_stream_u<16, 1>(L, x, K, xq, x_scale, x_rowsum, stream);
    if (nkb <= 32) return launch_tl1_stream_u<16, 2>(L, x, K, xq, x_scale, x_rowsum, stream);
    if (nkb <= 48) return launch_tl1_stream_u<16, 3>(L, x, K, xq, x_scale, x_rowsum, stream);
    return launch_tl1_stream_u<16, 4>(L, x, K, xq, x_scale, x_rowsum, stream);
}

size_t tl2_mfma_lds_bytes(int M, int K) { return (size_t)kTl2MfmaTables + (size_t)M * (K + 16); }

int tl2_mfma_max_tokens(int K) {
    const int nblk = K / kTl2BlockK;
    if (nblk < 1) return 0;
    const int waves = nblk <= 4 ? 4 : nblk <= 16 ? 8 : 16;
    const size_t budget = 160 * 1024 - (size_t)2 * waves * 64 * 16 - 256;   // less the reduction buffers
    // past 32 blocks (three per wave) the staging registers allow 8 tokens per slice; past 48 blocks (row groups
    // in several batches) only LDS limits the slice
    for (int m = nblk > 32 ? 8 : kTl2MfmaMaxTokens; m >= 1; --m)
        if (tl2_mfma_lds_bytes(m, K) <= budget) return m;
    return 0;
}

bool tl2_mfma_quant_fits(int K) {
    // one token quantised inside: the fp32 row in registers, at most 9 float4 per thread of 16 waves (K <= 36864,
    // the 100B-class down projection's 33024 included: 106 registers, no stack; 16 float4 beside two batches of
    // weight words need a stack frame, and that kernel ran 2.5x slower than the quantiser followed by the kernel
    // that reads the codes)
    return tl2_mfma_max_tokens(K) >= 1 && K / 4 <= 9 * 64 * 16;
}

template <int WAVES, int U, int CH, int XV, bool MB = false>
hipError_t launch_mfma_kernel(const FusedLinears& L, const float* x, int8_t* xq, float* x_scale, int32_t* x_rowsum,
                              int M, int K, hipStream_t stream) {
    const size_t lds = tl2_mfma_lds_bytes(M, K);
    const void* kern = reinterpret_cast<const void*>(tl2_mfma_decode_kernel<WAVES, U, CH, XV, MB>);
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, 64 * WAVES, lds) != hipSuccess || occ <= 0) occ = 1;
    const int64_t max_g = (int64_t)device_cus() * occ;
    const int64_t rounds = (L.total + max_g - 1) / max_g;
    const dim3 grid((unsigned)((L.total + rounds - 1) / rounds)), block(64 * WAVES);
    hipLaunchKernelGGL((tl2_mfma_decode_kernel<WAVES, U, CH, XV, MB>), grid, block, lds, stream, L, x, xq, x_scale,
                       x_rowsum, M, K);
    return hipGetLastError();
}

template <int WAVES, int U>
hipError_t launch_mfma_cfg(const FusedLinears& L, const int8_t* xq, const float* x_scale, int M, int K,
                           hipStream_t stream) {
    constexpr int kWide = U >= 3 ? 3 : 6;      // the slices of three blocks per wave hold at most 8 tokens
    int8_t* q = const_cast<int8_t*>(xq);
    float* s = const_cast<float*>(x_scale);
    if (M <= 8) return launch_mfma_kernel<WAVES, U, 3, 0>(L, nullptr, q, s, nullptr, M, K, stream);
    return launch_mfma_kernel<WAVES, U, kWide, 0>(L, nullptr, q, s, nullptr, M, K, stream);
}

// One token quantised inside: XV float4 of the row per thread.
template <int WAVES, int U>
hipError_t launch_mfma_quant(const FusedLinears& L, const float* x, int8_t* xq, float* x_scale, int32_t* x_rowsum,
                             int K, hipStream_t stream) {
    const int xv = (K / 4 + 64 * WAVES - 1) / (64 * WAVES);
    if (xv <= 1) return launch_mfma_kernel<WAVES, U, 1, 1>(L, x, xq, x_scale, x_rowsum, 1, K, stream);
    if (xv <= 2) return launch_mfma_kernel<WAVES, U, 1, 2>(L, x, xq, x_scale, x_rowsum, 1, K, stream);
    if (xv <= 4) return launch_mfma_kernel<WAVES, U, 1, 4>(L, x, xq, x_scale, x_rowsum, 1, K, stream);
    return launch_mfma_kernel<WAVES, U, 1, 8>(L, x, xq, x_scale, x_rowsum, 1, K, stream);
}

// One token quantised inside, row groups in several batches (K past 48 blocks, K / 4 <= 9216).
hipError_t launch_mfma_quant_mb(const FusedLinears& L, const float* x, int8_t* xq, float* x_scale,
                                int32_t* x_rowsum, int K, hipStream_t stream) {
    if (K / 4 <= 8 * 64 * 16) return launch_mfma_kernel<16, 3, 1, 8, true>(L, x, xq, x_scale, x_rowsum, 1, K, stream);
    return launch_mfma_kernel<16, 3, 1, 9, true>(L, x, xq, x_scale, x_rowsum, 1, K, stream);
}

// One token, quantised inside (tl2_mfma_quant_fits(K)).
hipError_t launch_tl2_mfma_quant(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                                 int32_t* x_rowsum, hipStream_t stream) {
    const int nblk = K / kTl2BlockK;
    if (!tl2_mfma_quant_fits(K)) return hipErrorInvalidValue;
    if (nblk > kTl2MfmaMaxBlocks) return launch_mfma_quant_mb(L, x, xq, x_scale, x_rowsum, K, stream);
    if (nblk <= 4) return launch_mfma_quant<4, 1>(L, x, xq, x_scale, x_rowsum, K, stream);
    if (nblk <= 8) return launch_mfma_quant<4, 2>(L, x, xq, x_scale, x_rowsum, K, stream);
    if (nblk <= 12) return launch_mfma_quant<4, 3>(L, x, xq, x_scale, x_rowsum, K, stream);
    if (nblk <= 16) return launch_mfma_quant<8, 2>(L, x, xq, x_scale, x_rowsum, K, stream);
    if (nblk <= 32) return launch_mfma_quant<16, 2>(L, x, xq, x_scale, x_rowsum, K, stream);
    return launch_mfma_quant<16, 3>(L, x, xq, x_scale, x_rowsum, K, stream);
}

// Waves and blocks per wave: every block of a row has its wave.  Tokens go in slices that fit in LDS.
hipError_t launch_tl2_mfma_decode(const FusedLinears& L, const int8_t* xq, const float* x_scale, int M, int K,
                                  hipStream_t stream) {
    const int nblk = K / kTl2BlockK;
    const int mc = tl2_mfma_max_tokens(K);
    if (mc < 1) return hipErrorInvalidValue;
    for (int m0 = 0; m0 < M; m0 += mc) {
        const int m = M - m0 < mc ? M - m0 : mc;
        FusedLinears Ls = L;
        for (int i = 0; i < L.count; ++i) {
            Ls.y[i] = L.y[i] + (size_t)m0 * L.N[i];
            Ls.acc[i] = L.acc[i] ? L.acc[i] + (size_t)m0 * L.N[i] : nullptr;
        }
        const int8_t* xs = xq + (size_t)m0 * K;
        const float* ss = x_scale + m0;
        hipError_t e;
        if (nblk > kTl2MfmaMaxBlocks)
            e = launch_mfma_kernel<16, 3, 3, 0, true>(Ls, nullptr, const_cast<int8_t*>(xs), const_cast<float*>(ss),
                                                      nullptr, m, K, stream);
        else if (nblk <= 4) e = launch_mfma_cfg<4, 1>(Ls, xs, ss, m, K, stream);
        else if (nblk <= 8) e = launch_mfma_cfg<8, 1>(Ls, xs, ss, m, K, stream);
        else if (nblk <= 16) e = launch_mfma_cfg<8, 2>(Ls, xs, ss, m, K, stream);
        else if (nblk <= 32) e = launch_mfma_cfg<16, 2>(Ls, xs, ss, m, K, stream);
        else e = launch_mfma_cfg<16, 3>(Ls, xs, ss, m, K, stream);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_tl2_to_i2s(const void* const* packed, const int* N, void* const* i2s_out, int count, int K,
                             hipStream_t stream) {
    if (count < 1 || count > kMaxFused) return hipErrorInvalidValue;
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    const int nblk = three / kTl2BlockK, units = (K - three) / kSubK;
    TranscodeLinears T{};
    long long pairs = 0, rest_groups = 0;
    for (int i = 0; i < kMaxFused; ++i) {
        const int j = i < count ? i : 0;
        T.packed[i] = static_cast<const uint8_t*>(packed[j]);
        T.out[i] = static_cast<uint32_t*>(i2s_out[j]);
        T.N[i] = N[j];
        T.pstart[i] = i < count ? pairs : 0x7fffffffffffffffLL;
        T.rstart[i] = i < count ? rest_groups : 0x7fffffffffffffffLL;
        if (i < count) {
            const long long rgs = N[i] / kRowsPerGroup;
            pairs += rgs * (nblk / 2);
            rest_groups += (rgs * 64 * ((nblk & 1) + units) + kTcThreads - 1) / kTcThreads;
        }
    }
    T.pairs = pairs;
    // persistent pair groups: as many as fit at once (eight per CU), no more than there are pairs
    const long long cap = (long long)device_cus() * 8;
    T.pair_groups = (int)(pairs < cap ? pairs : cap);
    const long long groups = T.pair_groups + rest_groups;
    if (groups < 1) return hipSuccess;
    hipLaunchKernelGGL(tl2_to_i2s_kernel, dim3((unsigned)groups), dim3(kTcThreads), 0, stream, T, K);
    return hipGetLastError();
}

hipError_t launch_elut_tables(const int8_t* xq, int M, int K, int16_t* lut, int16_t* lut1, hipStream_t stream) {
    const int three = (K / kTl2BlockK) * kTl2BlockK;
    const size_t total = (size_t)M * (three / 3 + (K - three) / 2);
    const unsigned grid = (unsigned)std::min<size_t>(4096, (total + 255) / 256);
    hipLaunchKernelGGL(elut_tables_kernel, dim3(grid > 0 ? grid : 1), dim3(256), 0, stream, xq, M, K, lut, lut1);
    return hipGetLastError();
}

}  // namespace bitnet
