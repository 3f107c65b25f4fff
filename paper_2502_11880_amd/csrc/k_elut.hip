// ELUT mpGEMM for integer weights of other cardinalities (Appendix "Insight", Table 3, Algorithm "ELUT mpGEMM",
// Eq. 3): the weights come from a set of C consecutive integers, every group of g weights is one code, and the
// accumulation looks the code up in a table of the C^g possible group sums of the token's activations (with mirror
// consolidation for symmetric sets: the non-negative half of the table, an index and a sign, Eq. 5).
//
// Formats (codes as the oracle defines them):
//   c4g2  C = 4 {-2, -1, 0, 1},  g = 2: 4-bit code = 4 (w0 + 2) + (w1 + 2), 16 entries, 2 bits per weight
//   c5g2  C = 5 {-2, .., 2},     g = 2: 4-bit index |5 w0 + w1| (13 entries) + a sign plane, 2.5 bits per weight
//   c3g5  C = 3 {-1, 0, 1},      g = 5: one byte per group, index |sum_j 3^(4-j) w_j| (122 entries) in bits 0-6 and
//                                       the sign in bit 7, 1.6 bits per weight
// A 122-entry table does not fit the 16-byte table registers of the paper's CPU kernels (its register-length
// analysis stops ternary groups at g = 3); in GPU LDS it costs 244 bytes per group and token.
//
// Kernel (decode, up to 4 tokens per launch; 2 for c3g5).  A work group of 16 waves owns 16 RS consecutive weight
// rows (RS per wave) and walks K in blocks of 64 packed words per row: each lane owns word l of a row's block, and
// the block's tables are built in LDS by the whole group (one entry per thread at a time, from the block's
// activation codes staged in LDS) before the lanes look their groups up.  Table entry e of group p of token t
// sits at ((t E' + e) * GB + q) with q = (p mod GW) * 64 + p / GW, so the 64 lanes of a wave reading item i of
// their words touch 64 consecutive entries when their codes agree.  Each lane keeps one int32 sum per row and
// token; a wave reduction and the epilogue y = acc * beta / s_t finish each row.  The kernel instance builds the
// tables of exactly the launch's tokens, and the next block's words and codes are loaded while the current block's
// tables are built and read.
#include "bitnet_internal.hpp"

namespace bitnet {
namespace {

template <int F>
struct ElutFmt;
template <>
struct ElutFmt<kElutC4G2> {
    static constexpr int C = 4, G = 2, E = 16, EP = 16, GW = 8, MT = 4;
    static constexpr bool kMirror = false;
};
template <>
struct ElutFmt<kElutC5G2> {
    static constexpr int C = 5, G = 2, E = 13, EP = 16, GW = 8, MT = 4;
    static constexpr bool kMirror = true;
};
template <>
struct ElutFmt<kElutC3G5> {
    static constexpr int C = 3, G = 5, E = 122, EP = 128, GW = 4, MT = 2;
    static constexpr bool kMirror = true;
};

constexpr int kEW = 16;                  // waves per work group
constexpr int kEThreads = 64 * kEW;

// Weight j of every table entry e, as a compile-time table: the base-C digits of e offset by the set's minimum, or
// with mirroring the balanced base-C digits of e; weight 0 is the most significant digit.  A table entry is then a
// sum of the group's codes with constant coefficients.
template <int F>
struct DigitTable {
    int8_t d[ElutFmt<F>::E][ElutFmt<F>::G];
    constexpr DigitTable() : d{} {
        using T = ElutFmt<F>;
        for (int e = 0; e < T::E; ++e) {
            int v = e;
            for (int j = T::G - 1; j >= 0; --j) {
                int r = 0;
                if (T::kMirror) {
                    r = v % T::C;
                    if (r > T::C / 2) r -= T::C;
                    v = (v - r) / T::C;
                } else {
                    r = v % T::C - T::C / 2;
                    v /= T::C;
                }
                d[e][j] = (int8_t)r;
            }
        }
    }
};

// One launch serves every weight of a fused group (rows concatenated, each row's weight found by a scalar compare
// chain), since the tables depend only on the activation.  QX (one token): the work group quantises the fp32 row
// itself (Sec. 2.1): the row's absmax first (a pass over the row, L2-resident after the first work groups), then
// every block's codes from its fp32 values as the block is staged; work group 0 writes the codes, the scale and
// their sum, as the quantiser would.
template <int F, int RS, int MT, bool QX>
__global__ __launch_bounds__(kEThreads) void elut_generic_kernel(FusedLinears L, const float* __restrict__ x,
                                                                 const int8_t* __restrict__ xq,
                                                                 const float* __restrict__ x_scale, int M, int K,
                                                                 int8_t* __restrict__ xq_out, float* __restrict__ s_out,
                                                                 int32_t* __restrict__ rs_out) {
    using T = ElutFmt<F>;
    constexpr int GB = 64 * T::GW;                // groups per block
    constexpr int KB = GB * T::G;                 // weights per block
    constexpr int kTab = MT * T::EP * GB;         // int16 entries
    constexpr int kXw = MT * (KB / 4);            // 32-bit words of activation codes per block
    static_assert(kXw <= kEThreads, "one word of codes per thread and block");
    static_assert(!QX || MT == 1, "the fused quantiser takes one token");
    __shared__ int16_t tab[kTab];
    __shared__ __align__(16) int8_t xs[MT][KB];
    __shared__ float redf[kEW];
    __shared__ int redi[kEW];
    constexpr DigitTable<F> kDig{};

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int Gtot = K / T::G;                    // groups per row
    const int nblk = (Gtot + GB - 1) / GB;
    const int rows = L.total * kRowsPerGroup;     // rows of all the launch's weights
    const int row0 = blockIdx.x * (kEW * RS) + wave * RS;
    const size_t row_bytes = T::GW == 8 ? (size_t)K / 4 : (size_t)K / 5;   // index plane (c4g2, c5g2) or bytes

    // this wave's rows: weight, row within it, packed row and (c5g2) sign row; rows past the last are clamped
    // to it and never stored
    int rli[RS], rn[RS];
    const uint8_t* rpk[RS];
    const uint8_t* rsg[RS];
#pragma unroll
    for (int r = 0; r < RS; ++r) {
        const int nc = min(row0 + r, rows - 1);
        int li, rg;
        locate(L, nc / kRowsPerGroup, li, rg);
        rli[r] = li;
        rn[r] = rg * kRowsPerGroup + nc % kRowsPerGroup;
        const uint8_t* base = pick(L.packed, li);
        rpk[r] = base + (size_t)rn[r] * row_bytes;
        rsg[r] = base + (size_t)pick(L.N, li) * K / 4 + (size_t)rn[r] * (K / 16);   // c5g2 only
    }

    // QX: the row's scale (the quantiser's formula) before the first block
    float sx = 1.0f;
    int csum = 0;                                 // QX, work group 0: this thread's share of the code sum
    if constexpr (QX) {
        const float4* x4 = reinterpret_cast<const float4*>(x);
        float amax = 0.0f;
        for (int i = tid; i < K / 4; i += kEThreads) {
            const float4 v = x4[i];
            amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v.x), fabsf(v.y)), fmaxf(fabsf(v.z), fabsf(v.w))));
        }
        amax = wave_max_all(amax);
        if (lane == 0) redf[wave] = amax;
        __syncthreads();
        amax = redf[0];
#pragma unroll
        for (int w = 1; w < kEW; ++w) amax = fmaxf(amax, redf[w]);
        sx = 127.0f / fmaxf(amax, 1e-5f);
    }

    // The loads of block kb: this wave's packed words (lane l: word l of each of its rows) and one word of the
    // block's activation codes per thread (token tid / (KB/4)), or with QX the float4 it quantises.  Addresses are
    // clamped to real words and the values past the block, the rows or the tokens zeroed, so every load is
    // unconditional.
    auto load_block = [&](int kb, uint32_t (&wv)[RS], uint32_t (&sv)[RS], uint32_t& xv, float4& xf) {
        const int gin = min(GB, Gtot - kb * GB);
        const int words = (gin + T::GW - 1) / T::GW;
        const int kin = gin * T::G;
        const int l = min(lane, words - 1);
#pragma unroll
        for (int r = 0; r < RS; ++r) {
            const bool ok = row0 + r < rows && lane < words;
            const uint32_t w = *reinterpret_cast<const uint32_t*>(rpk[r] + (size_t)kb * 256 + 4 * l);
            wv[r] = ok ? w : 0u;
            if constexpr (F == kElutC5G2) {
                const uint32_t sg = rsg[r][(size_t)kb * 64 + l];
                sv[r] = ok ? sg : 0u;
            } else {
                sv[r] = 0u;
            }
        }
        const int t = tid / (KB / 4), w = tid - t * (KB / 4);
        const bool xok = tid < kXw && t < M && 4 * w < kin;
        const size_t off = (size_t)kb * KB + min(4 * w, kin - 4);
        if constexpr (QX) {
            const float4 v = *reinterpret_cast<const float4*>(x + off);
            xf = xok ? v : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            xv = 0u;
        } else {
            const uint32_t v = *reinterpret_cast<const uint32_t*>(xq + (size_t)min(t, M - 1) * K + off);
            xv = xok ? v : 0u;
        }
    };

    int acc[RS][MT];
#pragma unroll
    for (int r = 0; r < RS; ++r)
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[r][t] = 0;

    // Block kb + 1's loads are issued before block kb's tables are built, so they land during its arithmetic.
    uint32_t wn[RS], sn[RS], xn;
    float4 xfn;
    load_block(0, wn, sn, xn, xfn);
    for (int kb = 0; kb < nblk; ++kb) {
        uint32_t wv[RS], sv[RS];
#pragma unroll
        for (int r = 0; r < RS; ++r) {
            wv[r] = wn[r];
            sv[r] = sn[r];
        }
        uint32_t xv = xn;
        if constexpr (QX) {
            // the block's codes from its fp32 values (zeros past the block quantise to zero codes)
            xv = quant4(xfn, sx);
            if (blockIdx.x == 0 && tid < kXw) {
                const int kin = min(GB, Gtot - kb * GB) * T::G;
                if (4 * tid < kin) {
                    reinterpret_cast<uint32_t*>(xq_out + (size_t)kb * KB)[tid] = xv;
                    csum = byte_sum4(xv, csum);
                }
            }
        }
        const int gin = min(GB, Gtot - kb * GB);             // groups in this block
        const int words = (gin + T::GW - 1) / T::GW;         // packed words per row in this block
        // 1. the block's activation codes into LDS (after every wave is done with the previous block's tables)
        __syncthreads();
        if (tid < kXw) reinterpret_cast<uint32_t*>(&xs[0][0])[tid] = xv;
        load_block(min(kb + 1, nblk - 1), wn, sn, xn, xfn);
        __syncthreads();
        // 2. the tables: one thread per token and group reads the group's codes once and writes all its entries,
        //    entry e = sum_j d_j(e) a_j with the digits as constants (groups past the block give zeros)
        for (int i = tid; i < MT * GB; i += kEThreads) {
            const int q = i % GB, t = i / GB;
            const int p = (q % 64) * T::GW + q / 64;
            int a[T::G];
#pragma unroll
            for (int j = 0; j < T::G; ++j) a[j] = p < gin ? (int)xs[t][p * T::G + j] : 0;
            int16_t* col = tab + (size_t)t * T::EP * GB + q;
#pragma unroll
            for (int e = 0; e < T::E; ++e) {
                int v = 0;
#pragma unroll
                for (int j = 0; j < T::G; ++j) v += (int)kDig.d[e][j] * a[j];
                col[e * GB] = (int16_t)v;
            }
        }
        __syncthreads();
        // 3. lookups: item i of lane l's word is group l GW + i, at table column i 64 + l
        if (lane < words) {
#pragma unroll
            for (int r = 0; r < RS; ++r) {
#pragma unroll
                for (int i = 0; i < T::GW; ++i) {
                    int idx, m;
                    if constexpr (F == kElutC3G5) {
                        const uint32_t b = (wv[r] >> (8 * i)) & 0xFFu;
                        idx = (int)(b & 0x7Fu);
                        m = -(int)(b >> 7);
                    } else {
                        idx = (int)((wv[r] >> (4 * i)) & 0xFu);
                        m = F == kElutC5G2 ? -(int)((sv[r] >> i) & 1u) : 0;
                    }
                    const int col = i * 64 + lane;
#pragma unroll
                    for (int t = 0; t < MT; ++t) {
                        const int v = tab[(t * T::EP + idx) * GB + col];
                        acc[r][t] += (v + m) ^ m;            // Eq. 5: the sign bit widened to a mask
                    }
                }
            }
        }
    }
    // 4. every row's sum over the lanes, then the epilogue
#pragma unroll
    for (int r = 0; r < RS; ++r) {
        const int li = rli[r], n = rn[r], N = pick(L.N, li);
        const float beta = *pick(L.w_scale, li);
        float* y = pick(L.y, li);
        int32_t* acc_out = pick(L.acc, li);
#pragma unroll
        for (int t = 0; t < MT; ++t) {
            const int total = wave_sum_all(acc[r][t]);
            if (lane == 0 && row0 + r < rows && t < M) {
                y[(size_t)t * N + n] = (float)total * (beta / (QX ? sx : x_scale[t]));
                if (acc_out) acc_out[(size_t)t * N + n] = total;
            }
        }
    }
    if constexpr (QX) {
        if (blockIdx.x == 0) {
            csum = wave_sum_all(csum);
            if (lane == 0) redi[wave] = csum;
            __syncthreads();
            if (tid == 0) {
                int tot = 0;
#pragma unroll
                for (int w = 0; w < kEW; ++w) tot += redi[w];
                rs_out[0] = tot;
                s_out[0] = sx;
            }
        }
    }
}

// Packing: one thread per packed word of a row (c4g2 and c5g2: 8 groups, plus their sign byte; c3g5: 4 groups).
// Values outside the set are clamped into it.
template <int F>
__global__ __launch_bounds__(256) void pack_elut_words(const int8_t* __restrict__ Wq, int N, int K,
                                                       uint8_t* __restrict__ packed) {
    using T = ElutFmt<F>;
    const size_t wpr = (size_t)K / (T::G * T::GW);       // words per row
    const size_t d = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (d >= (size_t)N * wpr) return;
    const size_t n = d / wpr;
    const int w = (int)(d - n * wpr);
    const int8_t* src = Wq + n * (size_t)K + (size_t)w * T::G * T::GW;
    const int lo = -(T::C / 2), hi = T::C - 1 - T::C / 2;
    uint32_t word = 0u, sign = 0u;
    for (int i = 0; i < T::GW; ++i) {
        int v = 0;
        for (int j = 0; j < T::G; ++j) {
            const int wj = min(max((int)src[i * T::G + j], lo), hi);
            v = v * T::C + (T::kMirror ? wj : wj - lo);
        }
        const uint32_t idx = (uint32_t)(v < 0 ? -v : v);
        const uint32_t sg = v < 0 ? 1u : 0u;
        if constexpr (F == kElutC3G5) word |= (idx | (sg << 7)) << (8 * i);
        else word |= idx << (4 * i);
        sign |= sg << i;
    }
    const size_t row_bytes = T::GW == 8 ? (size_t)K / 4 : (size_t)K / 5;
    *reinterpret_cast<uint32_t*>(packed + n * row_bytes + 4 * (size_t)w) = word;
    if constexpr (F == kElutC5G2) packed[(size_t)N * K / 4 + n * (K / 16) + w] = (uint8_t)sign;
}

template <int F, int RS, int MT, bool QX>
hipError_t launch_elut_mt(const FusedLinears& L, const float* x, const int8_t* xq, const float* x_scale, int M, int K,
                          int8_t* xq_out, float* s_out, int32_t* rs_out, hipStream_t stream) {
    const int64_t rows = (int64_t)L.total * kRowsPerGroup;
    const dim3 grid((unsigned)((rows + kEW * RS - 1) / (kEW * RS))), block(kEThreads);
    hipLaunchKernelGGL((elut_generic_kernel<F, RS, MT, QX>), grid, block, 0, stream, L, x, xq, x_scale, M, K, xq_out,
                       s_out, rs_out);
    return hipGetLastError();
}

// Tokens in slices of up to T::MT per launch; the kernel instance builds tables for exactly the slice's tokens
// (1, 2 or 4).  With x given (one token) the launch quantises the row itself.
template <int F, int RS>
hipError_t launch_elut_rs(const FusedLinears& L, const float* x, const int8_t* xq, const float* x_scale, int M,
                          int K, int8_t* xq_out, float* s_out, int32_t* rs_out, hipStream_t stream) {
    using T = ElutFmt<F>;
    if (x) return launch_elut_mt<F, RS, 1, true>(L, x, nullptr, nullptr, 1, K, xq_out, s_out, rs_out, stream);
    for (int m0 = 0; m0 < M; m0 += T::MT) {
        const int mc = M - m0 < T::MT ? M - m0 : T::MT;
        FusedLinears Ls = L;
        for (int i = 0; i < L.count; ++i) {
            Ls.y[i] = L.y[i] + (size_t)m0 * L.N[i];
            Ls.acc[i] = L.acc[i] ? L.acc[i] + (size_t)m0 * L.N[i] : nullptr;
        }
        const int8_t* xs = xq + (size_t)m0 * K;
        hipError_t e;
        if (mc == 1) e = launch_elut_mt<F, RS, 1, false>(Ls, nullptr, xs, x_scale + m0, mc, K, nullptr, nullptr, nullptr, stream);
        else if (mc == 2 || T::MT < 4)
            e = launch_elut_mt<F, RS, 2, false>(Ls, nullptr, xs, x_scale + m0, mc, K, nullptr, nullptr, nullptr, stream);
        else
            e = launch_elut_mt<F, RS, (T::MT >= 4 ? 4 : 2), false>(Ls, nullptr, xs, x_scale + m0, mc, K, nullptr, nullptr,
                                                                   nullptr, stream);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <int F>
hipError_t launch_elut_fmt(const FusedLinears& L, const float* x, const int8_t* xq, const float* x_scale, int M, int K,
                           int8_t* xq_out, float* s_out, int32_t* rs_out, hipStream_t stream) {
    // rows per wave: the fewest that keep the launch within one work group per CU (up to 8 rows per wave), so the
    // grid uses as many CUs as the rows allow (rounding up to a power of two left up to half of them idle: the
    // 3B-class layer set at one token, C4G2 54.7 -> 48.2 us per step with 3 and 6 rows allowed)
    const int cus = device_cus();
    const int64_t rows = (int64_t)L.total * kRowsPerGroup;
    const int64_t rs_need = (rows + kEW * cus - 1) / (kEW * cus);
    switch (rs_need <= 1 ? 1 : rs_need >= 8 ? 8 : (int)rs_need) {
        case 1: return launch_elut_rs<F, 1>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
        case 2: return launch_elut_rs<F, 2>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
        case 3: return launch_elut_rs<F, 3>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
        case 4: return launch_elut_rs<F, 4>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
        case 5: return launch_elut_rs<F, 5>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
        case 6: return launch_elut_rs<F, 6>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
        case 7: return launch_elut_rs<F, 7>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
        default: return launch_elut_rs<F, 8>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
    }
}

template <int F>
hipError_t launch_pack_fmt(const int8_t* Wq, int N, int K, void* packed, hipStream_t stream) {
    using T = ElutFmt<F>;
    const size_t words = (size_t)N * K / (T::G * T::GW);
    hipLaunchKernelGGL((pack_elut_words<F>), dim3((unsigned)((words + 255) / 256)), dim3(256), 0, stream, Wq, N, K,
                       static_cast<uint8_t*>(packed));
    return hipGetLastError();
}

}  // namespace

hipError_t launch_elut_generic(int fmt, const FusedLinears& L, const float* x, const int8_t* xq,
                               const float* x_scale, int M, int K, int8_t* xq_out, float* s_out, int32_t* rs_out,
                               hipStream_t stream) {
    switch (fmt) {
        case kElutC4G2: return launch_elut_fmt<kElutC4G2>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
        case kElutC5G2: return launch_elut_fmt<kElutC5G2>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
        default: return launch_elut_fmt<kElutC3G5>(L, x, xq, x_scale, M, K, xq_out, s_out, rs_out, stream);
    }
}

hipError_t launch_pack_elut(int fmt, const int8_t* Wq, int N, int K, void* packed, hipStream_t stream) {
    switch (fmt) {
        case kElutC4G2: return launch_pack_fmt<kElutC4G2>(Wq, N, K, packed, stream);
        case kElutC5G2: return launch_pack_fmt<kElutC5G2>(Wq, N, K, packed, stream);
        default: return launch_pack_fmt<kElutC3G5>(Wq, N, K, packed, stream);
    }
}

}  // namespace bitnet
